"""CPU oracle for the offline outlier-aware INT4 quantiser.

TEST INFRASTRUCTURE ONLY, like the rest of ``oracle/``: the library never
imports it and it imports nothing from the library.

Paper references (FlashQuant, arXiv 2608.15531):

* eq. (2) (Sec. 2.2, Outlier-Aware Quantization): q = round(w / s) + z with
  s = (w_max - w_min) / (2^b - 1) and z = round(-w_min / s); eq. (3):
  w_hat = s (q - z).
* Sec. 2.2: outliers are the high-magnitude weights, kept in bf16.
* Sec. 3.2.1: padding slots of the packed groups may hold original weights.

Readings where the paper is silent (kept in the design notes as well):

* b = 4, one (s, z) per group of 128 consecutive k of one column, over the
  group's non-outlier weights.
* The range is widened to contain 0 ([min(w_min, 0), max(w_max, 0)]) so that
  z lands in the unsigned code range; an all-zero group takes s = 1, z = 0.
* s is stored in fp16 as the smallest fp16 value not below the real s, and q
  and z are computed with that stored s; q and z are clamped to [0, 15].
* round() is round-half-to-even.
* Outliers: the round(frac K N) largest |w|, ties to the lower row-major index,
  among weights whose bf16 value is nonzero (bf16 zero marks a padding slot);
  their values are bf16(w) rounded to nearest even, and their codes are the
  group's zero-point so the dense part adds nothing there.
* Padding reuse: a padding slot whose tile-local position holds no real entry
  yet takes bf16(W[k, n]) if that is nonzero, and the code of (k, n) becomes the
  group's zero-point.

Parity status: pinned by hand-derived group constants (tests/golden), by the
closed form for weights already on an affine grid, by the rounding error bound
and by brute-force outlier selection.
"""

from __future__ import annotations

import numpy as np

from .oracle import bf16_rne_bits, bf16_to_f64, codes, f16_to_f64, zero_points

LEVELS = 15


def fp16_not_below(s: float) -> int:
    """Bit pattern of the smallest fp16 value >= s (0 < s <= 65504)."""
    h = np.float16(s)                     # nearest fp16, ties to even
    if float(h) < s:
        h = np.nextafter(h, np.float16(np.inf), dtype=np.float16)
    return int(np.array(h, dtype=np.float16).view(np.uint16))


def group_params(w: np.ndarray) -> tuple[int, int]:
    """(fp16 bits of s, z) of eq. (2) for one group's non-outlier weights."""
    lo = min(float(w.min()) if w.size else 0.0, 0.0)
    hi = max(float(w.max()) if w.size else 0.0, 0.0)
    s = (hi - lo) / LEVELS
    if s == 0.0:
        return 0x3C00, 0
    sb = fp16_not_below(s)
    s16 = float(f16_to_f64(np.array([sb], np.uint16))[0])
    z = int(np.clip(np.rint(-lo / s16), 0, LEVELS))
    return sb, z


def select_outliers(W: np.ndarray, frac: float) -> np.ndarray:
    """Row-major indices of the outliers, ascending."""
    K, N = W.shape
    flat = W.astype(np.float64).ravel()
    ok = (bf16_rne_bits(flat) & 0x7FFF) != 0
    idx = np.nonzero(ok)[0]
    want = min(int(np.round(frac * K * N)), idx.size)  # np.round: ties to even
    # sort by |w| descending, then index ascending
    order = np.lexsort((idx, -np.abs(flat[idx])))
    return np.sort(idx[order[:want]])


def quantize(W: np.ndarray, frac: float, group: int = 128):
    """eq. (2) per (group, column) plus bf16 outliers.
    Returns Wq, scales (fp16 bits), zeros, k, n, v (bf16 bits)."""
    W = np.asarray(W, dtype=np.float32)
    K, N = W.shape
    G = K // group
    sel = select_outliers(W, frac)
    is_out = np.zeros(K * N, bool)
    is_out[sel] = True
    is_out = is_out.reshape(K, N)
    q = np.zeros((K, N), np.int64)
    scales = np.zeros((G, N), np.uint16)
    z_all = np.zeros((G, N), np.int64)
    for g in range(G):
        for n in range(N):
            col = W[g * group:(g + 1) * group, n].astype(np.float64)
            keep = ~is_out[g * group:(g + 1) * group, n]
            sb, z = group_params(col[keep])
            s16 = float(f16_to_f64(np.array([sb], np.uint16))[0])
            qc = np.clip(np.rint(col / s16) + z, 0, LEVELS).astype(np.int64)
            qc[~keep] = z
            q[g * group:(g + 1) * group, n] = qc
            scales[g, n] = sb
            z_all[g, n] = z
    Wq = np.zeros((K // 8, N), np.uint32)
    for j in range(8):
        Wq |= (q[j::8].astype(np.uint32) << np.uint32(4 * j))
    zeros = np.zeros((G, N // 8), np.uint32)
    for j in range(8):
        zeros |= (z_all[:, j::8].astype(np.uint32) << np.uint32(4 * j))
    k, n = np.divmod(sel, N)
    v = bf16_rne_bits(W.astype(np.float64).ravel()[sel]).astype(np.uint16)
    return Wq, scales, zeros, k.astype(np.int32), n.astype(np.int32), v


def fill_padding(W: np.ndarray, group: int, tc, Wq: np.ndarray, zeros: np.ndarray,
                 k_tile: int = 128, n_tile: int = 64) -> int:
    """Padding reuse on an oracle TileCOO (packed and Wq updated in place)."""
    W = np.asarray(W, dtype=np.float32)
    K, N = W.shape
    kt = K // k_tile
    z_all = zero_points(zeros, K // group, N)
    filled = 0
    for t in range(len(tc.tile_indptr) - 1):
        kb, nb = (t % kt) * k_tile, (t // kt) * n_tile
        g0, g1 = int(tc.tile_indptr[t]), int(tc.tile_indptr[t + 1])
        slots = []
        for g in range(g0, g1):
            w4 = [int(x) for x in tc.packed[4 * g:4 * g + 4]]
            for j in range(4):
                kl = (w4[0] >> (8 * j)) & 0xFF
                nl = (w4[1] >> (8 * j)) & 0xFF
                val = (w4[2 + j // 2] >> (16 * (j % 2))) & 0xFFFF
                slots.append((g, j, kl, nl, val))
        taken = {(kl, nl) for (_, _, kl, nl, val) in slots if val != 0}
        for (g, j, kl, nl, val) in slots:
            if val != 0 or (kl, nl) in taken:
                continue
            k, n = kb + kl, nb + nl
            b = int(bf16_rne_bits(np.array([float(W[k, n])]))[0])
            if b & 0x7FFF == 0:
                continue
            taken.add((kl, nl))
            word = 4 * g + 2 + j // 2
            sh = 16 * (j % 2)
            tc.packed[word] = (int(tc.packed[word]) & ~(0xFFFF << sh) & 0xFFFFFFFF) | (b << sh)
            zc = int(z_all[k // group, n])
            Wq[k // 8, n] = (int(Wq[k // 8, n]) & ~(15 << (4 * (k % 8))) & 0xFFFFFFFF) | \
                (zc << (4 * (k % 8)))
            filled += 1
    return filled


def reconstruct(Wq, scales, zeros, K: int, N: int, group: int, k, n, v) -> np.ndarray:
    """dequant(W_Q) + densify(W_O) in float64 (eq. 3 plus the outliers)."""
    q = codes(Wq, K, N).astype(np.float64)
    z = np.repeat(zero_points(zeros, K // group, N).astype(np.float64), group, axis=0)
    s = np.repeat(f16_to_f64(scales), group, axis=0)
    Wh = s * (q - z)
    np.add.at(Wh, (np.asarray(k), np.asarray(n)), bf16_to_f64(np.asarray(v, np.uint16)))
    return Wh
