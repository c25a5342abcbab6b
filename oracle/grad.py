"""Oracle of the LoRA backward of the training chunk (test infrastructure only).

The paper trains each agent's adapter in the background while the frozen base
serves (§2.2: adapters on a frozen base model; §4: training runs as bounded
background chunks). For one projection of the mixed-adapter step,

    y_t = x_t W^T + s_t (x_t A_a^T) B_a^T,      a = a_t the token's adapter,

the gradients of a loss L with upstream gradient dy = dL/dy are, with
u_t = x_t A_a^T and g_t = s_t dy_t B_a (both restricted to a's rank r_a):

    dB_a = sum over tokens t of a of  s_t dy_t^T u_t      [N, r_a]
    dA_a = sum over tokens t of a of  g_t^T x_t           [r_a, K]
    dx_t = dy_t W + g_t A_a                               [K]

W is frozen (no gradient). Tokens without an adapter (index -1 or out of
range) contribute only dy_t W to dx. Rows and columns at or past an adapter's
rank are zero. Everything is float64 on the exact bf16 inputs; the products
are numpy matmuls over the tokens of one adapter at a time.
"""
from __future__ import annotations

import numpy as np

from . import bf16_to_f64


def lora_grad(x, dy, W, A, B, ranks, adapter_idx, scale):
    """x [T,K], dy [T,N], W [N,K], A [n_ad,r_max,K], B [n_ad,N,r_max] as
    uint16 bf16 bits; ranks [n_ad] (None = r_max), adapter_idx [T], scale [T].
    Returns (dA [n_ad,r_max,K], dB [n_ad,N,r_max], dx [T,K]) in float64."""
    xf, dyf, Wf = bf16_to_f64(x), bf16_to_f64(dy), bf16_to_f64(W)
    Af, Bf = bf16_to_f64(A), bf16_to_f64(B)
    n_ad, r_max, K = Af.shape
    N = Bf.shape[1]
    idx = np.asarray(adapter_idx, dtype=np.int64)
    s = np.asarray(scale, dtype=np.float64)
    rk = (np.full(n_ad, r_max) if ranks is None else
          np.clip(np.asarray(ranks, dtype=np.int64), 0, r_max))
    dA = np.zeros((n_ad, r_max, K))
    dB = np.zeros((n_ad, N, r_max))
    dx = dyf @ Wf
    for a in range(n_ad):
        rows = np.nonzero(idx == a)[0]
        r = int(rk[a])
        if rows.size == 0 or r == 0:
            continue
        sa = s[rows][:, None]
        u = xf[rows] @ Af[a, :r].T            # [T_a, r]
        g = sa * (dyf[rows] @ Bf[a, :, :r])   # [T_a, r]
        dB[a, :, :r] = dyf[rows].T @ (sa * u)
        dA[a, :r, :] = g.T @ xf[rows]
        dx[rows] += g @ Af[a, :r]
    return dA, dB, dx
