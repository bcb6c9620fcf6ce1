"""Oracle of the weight quantiser.  Test infrastructure only: tests, the smoke
check and the bench's CPU baseline use it; the library never does.

Definition (the symmetric form of the uniform quantiser of Section 2.2,
Eq. 1, in the format the MARLIN kernel decodes, with the group-wise clipping
search named in Section 3.5):

* A group is v = W[j*g : (j+1)*g, n], g consecutive rows of column n
  (g = K: the whole column).
* For a clipping ratio r the group's range is [-a, a] with a = r * max|v|;
  its 15 steps give the scale s = fp16(2a / 15), stored in fp16; the fixed
  zero point is 8 and the code of v is q = clamp(rint(v * (1/s)) + 8, 0, 15)
  (rint rounds half to even).  A scale that rounds to 0 gives every code 8.
* The reconstruction error of Section 2.2, e(r) = sum over the group of
  (v - s (q - 8))^2, is evaluated for every ratio in the caller's order; the
  group keeps the first ratio with the smallest error.

Precision: the codes and the choice of ratio are integer decisions taken by
floating-point arithmetic, so this oracle takes them in the kernel's
precision, fp32, in the order written above: each operation rounded on its
own (no fused multiply-add), and the error summed over the group's rows in
row order.  The ratios are the caller's fp32 values.
"""
from __future__ import annotations

import numpy as np

_F = np.float32


def _codes(v, sf, inv):
    """Code offsets t = q - 8 (fp32) of v for scale sf (0 -> every t = 0)."""
    t = np.clip(np.rint(v * inv), _F(-8), _F(7))
    return np.where(sf == 0, _F(0), t)


def quantize(W, group, ratios):
    """W float16 [K, N] -> (q uint8 [K, N], s float16 [G, N])."""
    W = np.asarray(W)
    assert W.dtype == np.float16 and W.ndim == 2
    K, N = W.shape
    g = K if group in (-1, None, K) else int(group)
    assert K % g == 0
    G = K // g
    V = W.astype(_F).reshape(G, g, N)  # V[j, k, n]: row k of group j, column n
    rs = np.asarray(ratios, dtype=_F).ravel()
    assert rs.size >= 1

    amax = np.abs(V).max(axis=1)  # [G, N]
    best_err = np.full((G, N), np.inf, dtype=_F)
    best = np.zeros((G, N), dtype=np.float16)
    with np.errstate(divide="ignore"):
        for r in rs:
            a = r * amax
            s16 = ((a + a) / _F(15)).astype(np.float16)
            sf = s16.astype(_F)
            inv = np.where(sf == 0, _F(0), _F(1) / sf)
            err = np.zeros((G, N), dtype=_F)
            for k in range(g):  # the group's rows, in order
                v = V[:, k, :]
                d = v - _codes(v, sf, inv) * sf
                err = err + d * d
            better = err < best_err
            best_err = np.where(better, err, best_err)
            best = np.where(better, s16, best)

        sf = best.astype(_F)
        inv = np.where(sf == 0, _F(0), _F(1) / sf)
    t = _codes(V, sf[:, None, :], inv[:, None, :])
    q = (t + _F(8)).astype(np.uint8).reshape(K, N)
    return q, best


def group_errors_f64(W, group, q, s):
    """Reconstruction error per group, sum (v - s (q - 8))^2, in float64."""
    W = np.asarray(W, dtype=np.float64)
    K, N = W.shape
    g = K if group in (-1, None, K) else int(group)
    G = K // g
    deq = np.repeat(np.asarray(s, dtype=np.float64), g, axis=0) * (np.asarray(q, dtype=np.float64) - 8.0)
    return ((W - deq) ** 2).reshape(G, g, N).sum(axis=1)
