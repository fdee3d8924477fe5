"""Training gradients of OctreeNCA -- TEST INFRASTRUCTURE ONLY.

The paper trains the whole OctreeNCA end to end by backpropagation through
every NCA step of every level, each level with its own weights (Sec. 3.2,
"Efficient Training of OctreeNCA"; supplement S7, training details).  This
module is the plain reference for that gradient: the derivative of a scalar
loss with respect to the five weight tensors of every level, obtained by the
chain rule through the steps of ``octree_nca`` taken in reverse order.  Only
``tests/`` and the benchmark's CPU-baseline leg may import it; the HIP
library never calls it and shares no code with it.

Arithmetic is float64.  The forward states are those of ``octree_nca``
(rounded to the storage type after every step); the backward takes each
stored state as the input of the next step and passes gradients straight
through the rounding, as automatic differentiation does through a cast.

Per step (state S -> S' = S + m * u on the hidden channels, Sec. 3.1), with
G' = dL/dS' and, recomputed from S, the perception P, f = [S, P],
a = W1 f + b1, h = ReLU(a), the fire bit m:

* gu[c] = m * G'[c] for hidden channels c >= n_in, 0 for input channels;
* dW2 += gu h^T;  gh = W2^T gu;  ga = gh * [a > 0] (ReLU' = 0 at 0);
* dW1 += ga f^T;  db1 += ga;  gf = W1^T ga = [gS, gP];
* dconv_b += gP;  dK[c, t] += gP[p, c] * S[p + o_t, c] (zero outside);
* dL/dS[q, c] = G'[q, c] + gS[q, c] + sum_t K[c, t] * gP[q - o_t, c].

Between levels the upsample copies each coarse cell to its children and the
level's image overwrites the input channels, so the coarse gradient of a
hidden channel is the sum over the children and the input channels get none.

Pins (tests/test_oracle_train.py): central finite differences of the forward
in float64 storage, the gradients of an independently written layer-wise
PyTorch forward (torch.autograd, float64, CPU), the adjoint identity of the
upsample, and the invariants fire rate 0 => zero weight gradients and
dL/dS = G'.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import List, Sequence, Tuple

import numpy as np

from .octree_nca import (build_pyramid, fire_bits, init_state, linear_index, nca_step, perceive,
                         tap_offsets, upsample_inject)


@dataclass
class LevelGrads:
    """Gradients of one level's weights, in the layouts of the weights."""
    conv_w: np.ndarray   # [C][taps]
    conv_b: np.ndarray   # [C]
    w1: np.ndarray       # [H][2C]
    b1: np.ndarray       # [H]
    w2: np.ndarray       # [C][H]

    @staticmethod
    def zeros(weights) -> "LevelGrads":
        return LevelGrads(*(np.zeros(np.shape(getattr(weights, k)), np.float64)
                            for k in ("conv_w", "conv_b", "w1", "b1", "w2")))

    def add(self, other: "LevelGrads") -> None:
        for k in ("conv_w", "conv_b", "w1", "b1", "w2"):
            getattr(self, k)[...] += getattr(other, k)


def _shift(x: np.ndarray, o: Tuple[int, int, int]) -> np.ndarray:
    """y[p] = x[p + o] with zeros where p + o falls outside x (first three axes)."""
    y = np.zeros_like(x)
    src, dst = [], []
    for n, off in zip(x.shape[:3], o):
        if off >= 0:
            src.append(slice(off, n)); dst.append(slice(0, n - off))
        else:
            src.append(slice(0, n + off)); dst.append(slice(-off, n))
    y[tuple(dst)] = x[tuple(src)]
    return y


def step_vjp(state: np.ndarray, weights, n_in: int, ndim: int, level: int, step: int, seed: int,
             fire_rate: float, g_out: np.ndarray, batch: int = 0):
    """Vector-Jacobian product of one NCA step at ``state`` (a whole level):
    returns (dL/dS, LevelGrads) for dL/dS' = ``g_out``."""
    s = np.asarray(state, np.float64)
    g_out = np.asarray(g_out, np.float64)
    d, h, w, c = s.shape
    kw = np.asarray(weights.conv_w, np.float64)
    w1 = np.asarray(weights.w1, np.float64)
    b1 = np.asarray(weights.b1, np.float64)
    w2 = np.asarray(weights.w2, np.float64)

    # recompute the forward activations of the step
    p = perceive(s, weights.conv_w, weights.conv_b, ndim)
    f = np.concatenate([s, p], axis=-1).reshape(-1, 2 * c)
    a = f @ w1.T + b1
    hid = np.maximum(a, 0.0)
    idx = linear_index((0, 0, 0), (d, h, w), (d, h, w))
    m = fire_bits(seed, level, step, idx, fire_rate, batch).astype(np.float64).reshape(-1)

    gu = np.zeros((d * h * w, c))
    gu[:, n_in:] = m[:, None] * g_out.reshape(-1, c)[:, n_in:]
    grads = LevelGrads.zeros(weights)
    grads.w2[...] = gu.T @ hid
    ga = (gu @ w2) * (a > 0.0)
    grads.w1[...] = ga.T @ f
    grads.b1[...] = ga.sum(axis=0)
    gf = ga @ w1
    g_s = gf[:, :c].reshape(s.shape)
    g_p = gf[:, c:].reshape(s.shape)
    grads.conv_b[...] = g_p.reshape(-1, c).sum(axis=0)
    g_in = g_out + g_s
    for t, o in enumerate(tap_offsets(ndim)):
        grads.conv_w[:, t] = (g_p * _shift(s, o)).reshape(-1, c).sum(axis=0)
        g_in += kw[:, t] * _shift(g_p, (-o[0], -o[1], -o[2]))
    return g_in, grads


def level_states(state: np.ndarray, weights, n_in: int, ndim: int, level: int, steps: int,
                 seed: int, fire_rate: float, dtype, batch: int = 0) -> List[np.ndarray]:
    """The states before each step and after the last: [S_0, S_1, ..., S_steps]."""
    out = [np.asarray(state, dtype)]
    for t in range(steps):
        out.append(nca_step(out[-1], weights, n_in, ndim, level, t, seed, fire_rate, dtype,
                            batch=batch))
    return out


def level_vjp(states: Sequence[np.ndarray], weights, n_in: int, ndim: int, level: int, seed: int,
              fire_rate: float, g_out: np.ndarray, batch: int = 0):
    """Backward through the steps of one level in reverse; ``states`` holds
    the state before each step (at least ``steps`` entries).  Returns (dL/dS_0,
    LevelGrads summed over the steps)."""
    grads = LevelGrads.zeros(weights)
    g = np.asarray(g_out, np.float64)
    for t in range(len(states) - 1, -1, -1):
        g, gt = step_vjp(states[t], weights, n_in, ndim, level, t, seed, fire_rate, g, batch)
        grads.add(gt)
    return g, grads


def upsample_vjp(g_fine: np.ndarray, factor: Sequence[int], n_in: int) -> np.ndarray:
    """Adjoint of the upsample + inject: each coarse hidden channel collects the
    sum of its children's gradients; input channels (overwritten by the image)
    get none."""
    fz, fy, fx = factor
    d, h, w, c = g_fine.shape
    g = np.asarray(g_fine, np.float64).reshape(d // fz, fz, h // fy, fy, w // fx, fx, c)
    coarse = g.sum(axis=(1, 3, 5))
    coarse[..., :n_in] = 0.0
    return coarse


@dataclass
class Tape:
    """Forward record of a training pass: per level (index = level), the states
    before each step and after the last."""
    states: List[List[np.ndarray]]

    @property
    def final(self) -> np.ndarray:
        return self.states[0][-1]


def train_forward(image: np.ndarray, weights: Sequence, *, ndim: int, n_in: int, channels: int,
                  factors: Sequence[Sequence[int]], steps: Sequence[int], fire_rate: float,
                  seed: int, dtype, batch: int = 0) -> Tape:
    """The inference of ``octree_nca.infer`` keeping every level's states."""
    levels = len(steps)
    pyr = build_pyramid(image, factors, dtype)
    state = init_state(pyr[-1], channels, dtype)
    per_level: List[List[np.ndarray]] = [[] for _ in range(levels)]
    for lvl in range(levels - 1, -1, -1):
        if lvl < levels - 1:
            state = upsample_inject(state, factors[lvl], pyr[lvl], dtype)
        per_level[lvl] = level_states(state, weights[lvl], n_in, ndim, lvl, steps[lvl], seed,
                                      fire_rate, dtype, batch)
        state = per_level[lvl][-1]
    return Tape(per_level)


def train_backward(tape: Tape, weights: Sequence, *, ndim: int, n_in: int,
                   factors: Sequence[Sequence[int]], seed: int, fire_rate: float,
                   g_final: np.ndarray, batch: int = 0) -> List[LevelGrads]:
    """Gradients of every level's weights for dL/dS_final = ``g_final``,
    backward from the finest level to the coarsest (whose seed carries no
    gradient further)."""
    levels = len(tape.states)
    grads: List[LevelGrads] = [None] * levels
    g = np.asarray(g_final, np.float64)
    for lvl in range(levels):
        st = tape.states[lvl][:-1]
        g, grads[lvl] = level_vjp(st, weights[lvl], n_in, ndim, lvl, seed, fire_rate, g, batch)
        if lvl < levels - 1:
            g = upsample_vjp(g, factors[lvl], n_in)
    return grads


def readout_mse(state: np.ndarray, target: np.ndarray):
    """Synthetic training loss on the readout channels (the last two, Sec. 3.2):
    L = 1/2 * sum over cells of sum over those channels of (S - Y)^2, with
    ``target`` Y of shape [D][H][W][2].  Returns (L, dL/dS)."""
    s = np.asarray(state, np.float64)
    diff = s[..., -2:] - np.asarray(target, np.float64)
    g = np.zeros_like(s)
    g[..., -2:] = diff
    return 0.5 * float(np.sum(diff * diff)), g
