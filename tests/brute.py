"""Brute-force, cell-by-cell restatements of the method with Python floats.

Used only on tiny grids to pin the oracle: each function follows the paper's
definition for a single cell with explicit loops, sharing nothing with the
oracle's vectorised code except the fire bits (pinned on their own against
numpy's Philox).
"""
import numpy as np

from oracle import fire_mask

C, H = 16, 64


def brute_pool(img, f):
    d, h, w, c = img.shape
    fz, fy, fx = f
    out = np.zeros((d // fz, h // fy, w // fx, c), dtype=np.float64)
    for z in range(d // fz):
        for y in range(h // fy):
            for x in range(w // fx):
                for ch in range(c):
                    acc = 0.0
                    for a in range(fz):
                        for b in range(fy):
                            for e in range(fx):
                                acc += float(img[fz * z + a, fy * y + b, fx * x + e, ch])
                    out[z, y, x, ch] = acc / (fz * fy * fx)
    return out.astype(img.dtype)


def brute_upsample(coarse, f, fine_img):
    d, h, w, n_in = fine_img.shape
    out = np.zeros((d, h, w, coarse.shape[-1]), dtype=coarse.dtype)
    for z in range(d):
        for y in range(h):
            for x in range(w):
                for ch in range(coarse.shape[-1]):
                    out[z, y, x, ch] = fine_img[z, y, x, ch] if ch < n_in else \
                        coarse[z // f[0], y // f[1], x // f[2], ch]
    return out


def brute_step(state, w, n_in, ndim, level, t, seed, fire_rate, dtype=np.float32):
    """One step, cell by cell, with Python floats (float64).  C and H are read
    from the weights' shapes."""
    C, H = w.conv_w.shape[0], w.w1.shape[0]
    d, h, wd, _ = state.shape
    mask = fire_mask(seed, level, t, (d, h, wd), fire_rate)
    out = np.array(state, dtype=np.float64)
    zs = (-1, 0, 1) if ndim == 3 else (0,)
    for z in range(d):
        for y in range(h):
            for x in range(wd):
                feat = [float(state[z, y, x, c]) for c in range(C)]
                for c in range(C):
                    acc = float(w.conv_b[c])
                    k = 0
                    for dz in zs:
                        for dy in (-1, 0, 1):
                            for dx in (-1, 0, 1):
                                zz, yy, xx = z + dz, y + dy, x + dx
                                if 0 <= zz < d and 0 <= yy < h and 0 <= xx < wd:
                                    acc += float(w.conv_w[c, k]) * float(state[zz, yy, xx, c])
                                k += 1
                    feat.append(acc)
                hid = []
                for j in range(H):
                    a = float(w.b1[j]) + sum(float(w.w1[j, i]) * feat[i] for i in range(2 * C))
                    hid.append(a if a > 0 else 0.0)
                if mask[z, y, x]:
                    for c in range(n_in, C):
                        out[z, y, x, c] += sum(float(w.w2[c, j]) * hid[j] for j in range(H))
    return out.astype(dtype)


def brute_infer(image, weights, ndim, n_in, factors, steps, fire_rate, seed, dtype=np.float32):
    pyr = [image]
    for f in factors:
        pyr.append(brute_pool(pyr[-1], f))
    levels = len(steps)
    d, h, w, _ = pyr[-1].shape
    state = np.zeros((d, h, w, C), dtype=dtype)
    state[..., :n_in] = pyr[-1]
    for lvl in range(levels - 1, -1, -1):
        if lvl < levels - 1:
            state = brute_upsample(state, factors[lvl], pyr[lvl])
        for t in range(steps[lvl]):
            state = brute_step(state, weights[lvl], n_in, ndim, lvl, t, seed, fire_rate, dtype)
    seg = np.zeros(state.shape[:3], dtype=np.uint8)
    for idx in np.ndindex(*state.shape[:3]):
        seg[idx] = 1 if state[idx + (C - 1,)] > state[idx + (C - 2,)] else 0
    return state, seg
