"""CPU oracle for the fused outlier-aware W4A16 decode matmul.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import or run anything in this
package.  The library (``paper_2608_15531_amd``) never imports it, and this
package imports nothing from the library: the two share no code.  The only
common dependency is the seeded input generator in ``synth/``.

Everything here is plain NumPy in float64, written for readability rather
than speed.  Paper references (FlashQuant, arXiv 2608.15531):

* eq. (1)  (Introduction): Y = X * dequant(W_Q) + X * W_O.
* eq. (3)  (Sec. 2.2, Outlier-Aware Quantization): w_hat = s * (q - z).
* Sec. 3.2.1 and Table 1: the Tile-COO arrays tile_indptr / bucket_info /
  packed_outliers, and the storage formula of the "Storage Analysis" passage.
* Sec. 3.2.2: column reordering (sort columns by nonzero count, greedy
  min-heap over bucket loads) and element reordering (gid = floor(k/2) % 4,
  bucket-rotated circular gid order).
* Sec. 4.2 (and the decoding listing it describes): four outliers per 16-byte
  group, per-column padding to a multiple of four.

Readings of passages where the paper is silent or ambiguous are documented
beside the code that takes them (the same list is kept in the design notes).

Parity status: the dense part, the outlier part, their sum, and the Tile-COO
round trip are pinned by the CPU tests (closed forms, library-routine special
cases, brute force, exact-arithmetic cases).  The Tile-COO *byte layout* has
no printed example in the paper (its format and reordering figures are not
available), so the byte layout itself is "parity unpinned" against the paper;
it is pinned only by its structural invariants and by an independent second
implementation.
"""

from __future__ import annotations

import heapq
from dataclasses import dataclass

import numpy as np

BY_COLUMN = 0
BY_BUCKET = 1
REORDER_COLUMNS = 1
REORDER_ELEMENTS = 2


# --------------------------------------------------------------------------
# number formats
# --------------------------------------------------------------------------

def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns -> float64 (exact: bf16 is the top half of fp32)."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32).astype(np.float64)


def f16_to_f64(bits: np.ndarray) -> np.ndarray:
    """IEEE fp16 bit patterns -> float64 (exact)."""
    return np.asarray(bits, dtype=np.uint16).view(np.float16).astype(np.float64)


def bf16_rne_bits(y: np.ndarray) -> np.ndarray:
    """float64 -> bf16 bits, round to nearest, ties to even, in one rounding.

    bf16 keeps 8 significant bits.  Scale each value so that its last kept bit
    has weight one, round half-to-even, scale back, and read the bits off the
    (now exactly representable) float32 value.  Subnormals use the fixed
    2^-133 unit; values that round past the largest finite bf16 become inf.
    """
    y = np.asarray(y, dtype=np.float64)
    _, e = np.frexp(y)
    unit_exp = np.maximum(e - 8, -133)
    r = np.round(np.ldexp(y, -unit_exp))
    with np.errstate(over="ignore"):
        val = np.ldexp(r, unit_exp).astype(np.float32)
    return (val.view(np.uint32) >> np.uint32(16)).astype(np.uint16)


# --------------------------------------------------------------------------
# dense part: eq. (3) then the product of eq. (1)
# --------------------------------------------------------------------------

def codes(Wq: np.ndarray, K: int, N: int) -> np.ndarray:
    """INT4 codes q[k, n]: nibble k % 8 (bits 4*(k%8)..+3) of word Wq[k//8, n]."""
    Wq = np.asarray(Wq, dtype=np.uint32).reshape(K // 8, N)
    q = np.empty((K, N), dtype=np.uint8)
    for j in range(8):
        q[j::8, :] = (Wq >> np.uint32(4 * j)) & np.uint32(0xF)
    return q


def zero_points(zeros: np.ndarray, n_groups: int, N: int) -> np.ndarray:
    """INT4 zero-points z[g, n]: nibble n % 8 of word zeros[g, n//8]."""
    zw = np.asarray(zeros, dtype=np.uint32).reshape(n_groups, N // 8)
    z = np.empty((n_groups, N), dtype=np.uint8)
    for j in range(8):
        z[:, j::8] = (zw >> np.uint32(4 * j)) & np.uint32(0xF)
    return z


def dequant(Wq, scales, zeros, K: int, N: int, group: int,
            cols: np.ndarray | None = None) -> np.ndarray:
    """W_hat[k, n] = s[g, n] * (q[k, n] - z[g, n]),  g = k // group  (eq. 3).

    The group size along K is not stated in the paper; the workloads fix 128.
    Returns float64 [K][len(cols)] (all columns when cols is None).
    """
    q = codes(Wq, K, N)
    z = zero_points(zeros, K // group, N)
    s = f16_to_f64(np.asarray(scales).reshape(K // group, N))
    if cols is not None:
        q, z, s = q[:, cols], z[:, cols], s[:, cols]
    g_of_k = np.arange(K) // group
    return s[g_of_k, :] * (q.astype(np.float64) - z[g_of_k, :].astype(np.float64))


def dense_part(X, Wq, scales, zeros, K, N, group, cols=None, block=2048):
    """X * dequant(W_Q) in float64, blocked over output columns."""
    X64 = bf16_to_f64(X)
    cols = np.arange(N) if cols is None else np.asarray(cols)
    out = np.empty((X64.shape[0], cols.size), dtype=np.float64)
    for c0 in range(0, cols.size, block):
        cb = cols[c0:c0 + block]
        out[:, c0:c0 + cb.size] = X64 @ dequant(Wq, scales, zeros, K, N, group, cb)
    return out


# --------------------------------------------------------------------------
# outlier part: the sparse product of eq. (1)
# --------------------------------------------------------------------------

def outlier_part(X, k, n, v, N, cols=None):
    """X * W_O for W_O given as COO triples, by scatter-add in float64."""
    X64 = bf16_to_f64(X)
    k = np.asarray(k, dtype=np.int64)
    n = np.asarray(n, dtype=np.int64)
    v64 = bf16_to_f64(v)
    if cols is None:
        Y = np.zeros((X64.shape[0], N), dtype=np.float64)
        np.add.at(Y.T, n, (X64[:, k] * v64).T)
        return Y
    cols = np.asarray(cols, dtype=np.int64)
    where = np.full(N, -1, dtype=np.int64)
    where[cols] = np.arange(cols.size)
    sel = where[n] >= 0
    Y = np.zeros((X64.shape[0], cols.size), dtype=np.float64)
    np.add.at(Y.T, where[n[sel]], (X64[:, k[sel]] * v64[sel]).T)
    return Y


def matmul(X, Wq, scales, zeros, K, N, group, k, n, v, cols=None):
    """Y = X * dequant(W_Q) + X * W_O in float64 (eq. 1), optionally only cols."""
    return (dense_part(X, Wq, scales, zeros, K, N, group, cols)
            + outlier_part(X, k, n, v, N, cols))


def matmul_tile_coo(X, Wq, scales, zeros, K, N, group, tc: "TileCOO", cols=None):
    """eq. (1) with W_O read back through this oracle's own Tile-COO unpack."""
    k, n, v = unpack_tile_coo(K, N, tc.params, tc.tile_indptr, tc.bucket_info, tc.packed)
    return matmul(X, Wq, scales, zeros, K, N, group, k, n, v, cols)


# --------------------------------------------------------------------------
# Tile-COO (Sec. 3.2.1, Table 1; reordering Sec. 3.2.2; groups Sec. 4.2)
# --------------------------------------------------------------------------

@dataclass(frozen=True)
class Params:
    k_tile: int = 128          # K_SHM
    n_tile: int = 64           # N_SHM
    buckets: int = 16          # N_warp * N_bucket buckets per tile
    group_mode: int = BY_COLUMN
    reorder: int = REORDER_COLUMNS | REORDER_ELEMENTS
    elems_per_bank: int = 2    # gid = (k // elems_per_bank) % n_bank_groups
    n_bank_groups: int = 4


@dataclass
class TileCOO:
    params: Params
    tile_indptr: np.ndarray    # uint32 [n_tiles + 1], absolute group offsets
    bucket_info: np.ndarray    # uint16 [2 * n_tiles * buckets]: (offset, count)
    packed: np.ndarray         # uint32 [4 * n_groups]
    nnz: int

    @property
    def n_tiles(self) -> int:
        return int(self.tile_indptr.shape[0]) - 1

    @property
    def n_groups(self) -> int:
        return int(self.packed.shape[0]) // 4

    @property
    def n_buckets(self) -> int:
        return self.n_tiles * self.params.buckets

    @property
    def bytes(self) -> int:
        return storage_bytes(self.n_tiles, self.n_buckets, 4 * self.n_groups)


def storage_bytes(n_tiles: int, n_buckets: int, n_slots: int) -> int:
    """Tile-COO size (Storage Analysis, Sec. 3.2.1) with padded slots counted.

    4 bytes per tile_indptr entry (n_tiles + 1 of them), 4 bytes per bucket
    (two uint16), 4 bytes per stored slot (u8 row, u8 column, bf16 value).
    """
    return 4 * (n_tiles + 1) + 4 * n_buckets + 4 * n_slots


def csr_bytes(K: int, nnz: int) -> int:
    """CSR size as the paper counts it: (K+1) 4-byte pointers + 12 B per nonzero."""
    return 4 * (K + 1) + 12 * nnz


class FormatError(ValueError):
    pass


def check_params(K: int, N: int, p: Params) -> None:
    if not (1 <= p.k_tile <= 256 and 1 <= p.n_tile <= 256):
        raise FormatError("tile sides must be in 1..256 (u8 local indices)")
    if K % p.k_tile or N % p.n_tile:
        raise FormatError("K and N must be multiples of the tile sides")
    if not 1 <= p.buckets <= 1024:
        raise FormatError("buckets per tile must be in 1..1024")
    if p.group_mode not in (BY_COLUMN, BY_BUCKET):
        raise FormatError("unknown group mode")
    if p.reorder & ~3:
        raise FormatError("unknown reorder bits")
    if p.elems_per_bank < 1 or p.n_bank_groups < 1 or \
            p.elems_per_bank * p.n_bank_groups > p.k_tile:
        raise FormatError("gid parameters must satisfy epb * ngroups <= k_tile")


def check_coo(K: int, N: int, k, n, v) -> None:
    k = np.asarray(k, dtype=np.int64)
    n = np.asarray(n, dtype=np.int64)
    v = np.asarray(v, dtype=np.uint16)
    if not (k.shape == n.shape == v.shape):
        raise FormatError("COO arrays must have equal length")
    if k.size and (k.min() < 0 or k.max() >= K or n.min() < 0 or n.max() >= N):
        raise FormatError("COO index out of range")
    if k.size and np.unique(k * N + n).size != k.size:
        raise FormatError("duplicate COO position")
    if np.any((v & 0x7FFF) == 0):
        raise FormatError("zero-valued outlier (bits 0x0000 mark padding)")


def _bucket_columns(cols: list[int], counts: list[int], p: Params) -> list[list[int]]:
    """Assign a tile's nonempty columns to buckets; return each bucket's columns
    in processing order.

    Column reordering on (Sec. 3.2.2): sort columns by count, descending (ties
    by column index), then give each to the bucket with the smallest running
    count (ties by lowest bucket id); a bucket keeps its columns in assignment
    order.  The balance measure is the raw nonzero count.
    Column reordering off: the uniform column-wise split the paper argues
    against, bucket = column * buckets // n_tile, columns ascending.
    """
    buckets: list[list[int]] = [[] for _ in range(p.buckets)]
    if p.reorder & REORDER_COLUMNS:
        order = sorted(range(len(cols)), key=lambda i: (-counts[i], cols[i]))
        heap = [(0, b) for b in range(p.buckets)]
        for i in order:
            load, b = heapq.heappop(heap)
            buckets[b].append(cols[i])
            heapq.heappush(heap, (load + counts[i], b))
    else:
        for c in sorted(cols):
            buckets[c * p.buckets // p.n_tile].append(c)
    return buckets


def _gid(kl: int, p: Params) -> int:
    """Bank group of a row index (Sec. 3.2.2 element reordering; paper: floor(k/2) % 4)."""
    return (kl // p.elems_per_bank) % p.n_bank_groups


def _reorder_elements(elems: list[tuple], start_pos: int, rot: int, p: Params) -> list[tuple]:
    """Order elements so slot position pos reads bank group (pos + rot) % ngroups.

    elems: (kl, ...) tuples already sorted by their within-queue order.
    Each gid queue keeps that order.  When the target queue is empty the next
    non-empty queue in circular order is taken (the paper does not say what
    happens once a group runs out; this is our reading).
    """
    ng = p.n_bank_groups
    queues: list[list[tuple]] = [[] for _ in range(ng)]
    for e in elems:
        queues[_gid(e[0], p)].append(e)
    heads = [0] * ng
    out = []
    pos = start_pos
    for _ in range(len(elems)):
        t = (pos + rot) % ng
        for d in range(ng):
            qi = (t + d) % ng
            if heads[qi] < len(queues[qi]):
                out.append(queues[qi][heads[qi]])
                heads[qi] += 1
                break
        pos += 1
    return out


def _pad_slot(pos: int, rot: int, col: int, p: Params) -> tuple:
    """Pad slot: value bits 0x0000, row index chosen in the slot's target gid."""
    return (p.elems_per_bank * ((pos + rot) % p.n_bank_groups), col, 0)


def _bucket_slots(bucket_cols: list[int], tile_elems: dict, b: int, p: Params) -> list[tuple]:
    """Slot list (kl, nl, vbits) of one bucket, padded to a multiple of 4."""
    rot = b % p.n_bank_groups
    slots: list[tuple] = []
    if p.group_mode == BY_COLUMN:
        # Sec. 4.2: each column padded to a multiple of four so that the four
        # values of a 16-byte group share one column index.
        for c in bucket_cols:
            elems = sorted((kl, c, vb) for kl, vb in tile_elems[c])
            if p.reorder & REORDER_ELEMENTS:
                elems = _reorder_elements(elems, len(slots), rot, p)
            slots.extend(elems)
            while len(slots) % 4:
                slots.append(_pad_slot(len(slots), rot, c, p))
    else:
        # Sec. 3.2.1 Packed Outliers: groups of four per bucket, only the
        # bucket tail padded.  Within-queue order: (row, column position).
        colpos = {c: i for i, c in enumerate(bucket_cols)}
        elems = [(kl, c, vb) for c in bucket_cols for kl, vb in tile_elems[c]]
        if p.reorder & REORDER_ELEMENTS:
            elems.sort(key=lambda e: (e[0], colpos[e[1]]))
            elems = _reorder_elements(elems, 0, rot, p)
        else:
            elems.sort(key=lambda e: (colpos[e[1]], e[0]))
        slots.extend(elems)
        while len(slots) % 4:
            slots.append(_pad_slot(len(slots), rot, slots[-1][1], p))
    return slots


def _group_words(s4: list[tuple]) -> list[int]:
    """Four slots -> four little-endian uint32 words: rows, columns, values."""
    w0 = s4[0][0] | (s4[1][0] << 8) | (s4[2][0] << 16) | (s4[3][0] << 24)
    w1 = s4[0][1] | (s4[1][1] << 8) | (s4[2][1] << 16) | (s4[3][1] << 24)
    w2 = s4[0][2] | (s4[1][2] << 16)
    w3 = s4[2][2] | (s4[3][2] << 16)
    return [w0, w1, w2, w3]


def pack_tile_coo(K: int, N: int, k, n, v, p: Params = Params()) -> TileCOO:
    """Encode COO outliers into Tile-COO (Sec. 3.2.1, Table 1; Sec. 3.2.2).

    Readings taken where the paper is silent:
    * tile order is N-strip-major: t = (n // n_tile) * (K // k_tile) + k // k_tile;
    * bucket_info holds, per bucket, the offset of its first group relative to
      the start of its tile and its number of 16-byte groups (both uint16);
      buckets of a tile are stored contiguously in bucket order;
    * tile_indptr holds absolute group offsets;
    * a group stores four u8 rows, four u8 columns, four bf16 values.
    """
    check_params(K, N, p)
    check_coo(K, N, k, n, v)
    k = np.asarray(k, dtype=np.int64)
    n = np.asarray(n, dtype=np.int64)
    v = np.asarray(v, dtype=np.uint16)
    kt_count, nt_count = K // p.k_tile, N // p.n_tile
    n_tiles = kt_count * nt_count
    tile = (n // p.n_tile) * kt_count + (k // p.k_tile)
    kl = k % p.k_tile
    nl = n % p.n_tile
    order = np.argsort(tile, kind="stable")
    bounds = np.searchsorted(tile[order], np.arange(n_tiles + 1))

    tile_indptr = np.zeros(n_tiles + 1, dtype=np.uint32)
    bucket_info = np.zeros(2 * n_tiles * p.buckets, dtype=np.uint16)
    words: list[int] = []
    for t in range(n_tiles):
        idx = order[bounds[t]:bounds[t + 1]]
        tile_elems: dict[int, list] = {}
        for i in idx:
            tile_elems.setdefault(int(nl[i]), []).append((int(kl[i]), int(v[i])))
        cols = sorted(tile_elems)
        counts = [len(tile_elems[c]) for c in cols]
        buckets = _bucket_columns(cols, counts, p)
        tile_start = len(words) // 4
        tile_indptr[t] = tile_start
        for b in range(p.buckets):
            slots = _bucket_slots(buckets[b], tile_elems, b, p)
            off = len(words) // 4 - tile_start
            cnt = len(slots) // 4
            if off > 0xFFFF or cnt > 0xFFFF:
                raise FormatError("bucket offset or count exceeds uint16")
            bucket_info[2 * (t * p.buckets + b)] = off
            bucket_info[2 * (t * p.buckets + b) + 1] = cnt
            for g in range(cnt):
                words.extend(_group_words(slots[4 * g:4 * g + 4]))
    tile_indptr[n_tiles] = len(words) // 4
    return TileCOO(p, tile_indptr, bucket_info, np.array(words, dtype=np.uint32), int(k.size))


def unpack_tile_coo(K: int, N: int, p: Params, tile_indptr, bucket_info, packed):
    """Inverse of pack_tile_coo: walk tiles -> buckets -> groups -> slots, drop
    pad slots (value bits 0x0000), return (k, n, v) sorted by (k, n)."""
    tile_indptr = np.asarray(tile_indptr, dtype=np.int64)
    bucket_info = np.asarray(bucket_info, dtype=np.int64)
    packed = np.asarray(packed, dtype=np.uint32).reshape(-1, 4)
    kt_count = K // p.k_tile
    ks, ns, vs = [], [], []
    for t in range(tile_indptr.size - 1):
        k0 = (t % kt_count) * p.k_tile
        n0 = (t // kt_count) * p.n_tile
        for b in range(p.buckets):
            off = bucket_info[2 * (t * p.buckets + b)]
            cnt = bucket_info[2 * (t * p.buckets + b) + 1]
            g = packed[tile_indptr[t] + off: tile_indptr[t] + off + cnt]
            if g.size == 0:
                continue
            for j in range(4):
                kl = (g[:, 0] >> np.uint32(8 * j)) & np.uint32(0xFF)
                nl = (g[:, 1] >> np.uint32(8 * j)) & np.uint32(0xFF)
                vb = (g[:, 2 + j // 2] >> np.uint32(16 * (j % 2))) & np.uint32(0xFFFF)
                real = vb != 0
                ks.append(k0 + kl[real].astype(np.int64))
                ns.append(n0 + nl[real].astype(np.int64))
                vs.append(vb[real].astype(np.uint16))
    if not ks:
        return np.zeros(0, np.int64), np.zeros(0, np.int64), np.zeros(0, np.uint16)
    k, n, v = np.concatenate(ks), np.concatenate(ns), np.concatenate(vs)
    order = np.lexsort((n, k))
    return k[order], n[order], v[order]


def coo_sorted(k, n, v):
    """COO triples sorted by (k, n), for comparisons."""
    k = np.asarray(k, dtype=np.int64)
    n = np.asarray(n, dtype=np.int64)
    v = np.asarray(v, dtype=np.uint16)
    order = np.lexsort((n, k))
    return k[order], n[order], v[order]


def bank_group_collisions(tc: TileCOO, t: int, lanes_per_step: int | None = None) -> int:
    """Element-reordering metric: step the buckets of tile t in lockstep, one
    slot per bucket per step (one sub-wave per bucket, Sec. 3.2.2), and count
    at every step how many buckets read a bank group another bucket already
    reads.  Pad slots count as reads.  Lower is better."""
    p = tc.params
    nb = p.buckets if lanes_per_step is None else lanes_per_step
    base = int(tc.tile_indptr[t])
    info = tc.bucket_info.reshape(-1, 2)[t * p.buckets:(t + 1) * p.buckets]
    slots = []
    for b in range(p.buckets):
        off, cnt = int(info[b, 0]), int(info[b, 1])
        g = tc.packed.reshape(-1, 4)[base + off: base + off + cnt]
        ks = [(int(w) >> (8 * j)) & 0xFF for w in g[:, 0] for j in range(4)]
        slots.append(ks)
    total = 0
    for b0 in range(0, p.buckets, nb):
        group = slots[b0:b0 + nb]
        steps = max((len(s) for s in group), default=0)
        for step in range(steps):
            gids = [_gid(s[step], p) for s in group if step < len(s)]
            total += len(gids) - len(set(gids))
    return total
