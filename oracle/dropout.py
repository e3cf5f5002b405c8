"""Value dropout with per-slice seeds (Sec. 5: one seed per slice n, reused in
the forward and the backward pass through that slice).

TEST INFRASTRUCTURE ONLY, like the rest of oracle/.

Definition (the library's interface documents the same):
  * Philox4x64-10, the counter-based generator of Salmon et al., "Parallel
    random numbers: as easy as 1, 2, 3" (SC 2011): a 4 x 64-bit counter and
    a 2 x 64-bit key, ten rounds of two 64 x 64 -> 128-bit products with
    the multipliers 0xD2E7470EE14C6C93 and 0xCA5A826395121157, the key
    bumped by the Weyl constants 0x9E3779B97F4A7C15 and 0xBB67AE8584CAA73B
    between rounds;
  * value element (b, h, l, e) of a problem with H heads and slice length C
    lies in slice n = l // C at row r = l - n C; slice n's seed is the key
    (seed, n); the counter is (r, e // 16, b H + h, 0); the element reads
    16-bit field j = e % 16 of the four outputs (word j // 4, bits
    16 (j % 4) .. 16 (j % 4) + 15);
  * the element is kept when that field is >= t = round(p 65536) (so p = 0
    keeps everything), and the output is scaled by s = 1 / (1 - p):
        Y_l = s sum_{l' <= l} a_ll' (m_l' * V_l') / sum_{l' <= l} a_ll'.
"""

from __future__ import annotations

import numpy as np

_M0, _M1 = 0xD2E7470EE14C6C93, 0xCA5A826395121157
_W0, _W1 = 0x9E3779B97F4A7C15, 0xBB67AE8584CAA73B
_LO32 = np.uint64(0xFFFFFFFF)


def _mulhilo(a: int, b: np.ndarray):
    """(hi, lo) 64-bit halves of the 128-bit product of the constant a and
    the uint64 array b, from 32-bit limbs."""
    b = b.astype(np.uint64)
    a_lo, a_hi = np.uint64(a & 0xFFFFFFFF), np.uint64(a >> 32)
    b_lo, b_hi = b & _LO32, b >> np.uint64(32)
    ll = a_lo * b_lo
    lh = a_lo * b_hi
    hl = a_hi * b_lo
    hh = a_hi * b_hi
    mid = (ll >> np.uint64(32)) + (lh & _LO32) + (hl & _LO32)
    lo = (ll & _LO32) | ((mid & _LO32) << np.uint64(32))
    hi = hh + (lh >> np.uint64(32)) + (hl >> np.uint64(32)) + (mid >> np.uint64(32))
    return hi, lo


def philox4x64_10(ctr, key):
    """Philox4x64-10 of counters ctr (4 uint64 arrays, broadcast together)
    under keys key (2 uint64 arrays or ints).  Returns 4 uint64 arrays."""
    c0, c1, c2, c3 = (np.asarray(c, dtype=np.uint64) for c in ctr)
    k0, k1 = (np.asarray(k, dtype=np.uint64) for k in key)
    with np.errstate(over="ignore"):
        for _ in range(10):
            hi0, lo0 = _mulhilo(_M0, c0)
            hi1, lo1 = _mulhilo(_M1, c2)
            c0, c1, c2, c3 = hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0
            k0 = k0 + np.uint64(_W0)
            k1 = k1 + np.uint64(_W1)
    return c0, c1, c2, c3


def keep_threshold(p: float) -> int:
    if not (0.0 <= p < 1.0):
        raise ValueError("dropout probability must be in [0, 1)")
    return int(round(p * 65536.0))


def value_mask(B: int, H: int, L: int, d: int, C: int, p: float, seed: int) -> np.ndarray:
    """0/1 float64 mask [B, H, L, d] of the definition above."""
    t = keep_threshold(p)
    C = min(C, L)
    l = np.arange(L, dtype=np.uint64)
    n = l // np.uint64(C)
    r = l - n * np.uint64(C)
    e = np.arange(d)
    grp = (e // 16).astype(np.uint64)
    field = e % 16
    head = np.arange(B * H, dtype=np.uint64).reshape(B, H, 1, 1)
    shape = (B, H, L, len(np.unique(grp)))
    ctr = (np.broadcast_to(r[None, None, :, None], shape), np.broadcast_to(np.unique(grp)[None, None, None, :], shape),
           np.broadcast_to(head, shape), np.zeros(shape, dtype=np.uint64))
    key = (np.uint64(seed), np.broadcast_to(n[None, None, :, None], shape))
    words = np.stack(philox4x64_10(ctr, key), axis=-1)  # [B, H, L, groups, 4]
    w = words[:, :, :, grp, field // 4]  # [B, H, L, d]
    f = (w >> (16 * (field % 4)).astype(np.uint64)) & np.uint64(0xFFFF)
    return (f >= np.uint64(t)).astype(np.float64)


def output_scale(p: float) -> float:
    """s = 1 / (1 - p), rounded to float32 as the library applies it."""
    return float(np.float32(1.0 / (1.0 - p)))


def dropout_forward(attention_forward, Q, K, V, W, kind, C, p, seed, **kw):
    """Y = s * attention(Q, K, m * V) with the mask of the definition."""
    V = np.asarray(V.detach().cpu().double().numpy() if hasattr(V, "detach") else V, dtype=np.float64)
    B, H, L, d = V.shape
    m = value_mask(B, H, L, d, C, p, seed)
    return output_scale(p) * attention_forward(Q, K, m * V, W, kind, **kw)


def dropout_backward(attention_backward, Q, K, V, W, dY, kind, C, p, seed, **kw):
    """Gradients of sum(dY * Y) for Y = s * attention(Q, K, m * V): the
    attention's VJP at cotangent s dY, with dV masked by m."""
    V = np.asarray(V.detach().cpu().double().numpy() if hasattr(V, "detach") else V, dtype=np.float64)
    dY = np.asarray(dY.detach().cpu().double().numpy() if hasattr(dY, "detach") else dY, dtype=np.float64)
    B, H, L, d = V.shape
    m = value_mask(B, H, L, d, C, p, seed)
    s = output_scale(p)
    dQ, dK, dV, dW = attention_backward(Q, K, m * V, W, s * dY, kind, **kw)
    return dQ, dK, m * dV, dW
