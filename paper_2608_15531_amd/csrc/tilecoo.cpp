// Host-side Tile-COO encoder, decoder and validator.
//
// Format: FlashQuant Sec. 3.2.1 and Table 1 (tile_indptr, bucket_info,
// packed_outliers); offline reordering: Sec. 3.2.2 (column reordering by a
// greedy min-heap over bucket loads, element reordering by bank group);
// 16-byte groups of four slots padded per column: Sec. 4.2.
//
// Readings of the paper taken here (it is silent on them):
//   * tiles are numbered N-strip-major, t = (n / n_tile) * (K / k_tile) + k / k_tile,
//     so the tiles one output strip needs are contiguous;
//   * bucket_info offsets are in groups, relative to the tile's first group;
//     counts are in groups; buckets of a tile are stored in bucket order;
//   * columns are sorted by (count descending, column ascending) and heap ties
//     go to the lowest bucket id; without column reordering bucket
//     b holds the contiguous columns [b*n_tile/B, (b+1)*n_tile/B);
//   * element reordering targets bank group (pos + b) % n_bank_groups at slot
//     position pos of bucket b and falls through to the next non-empty bank
//     group, in circular order, once the target group is exhausted;
//   * a padding slot has value bits 0x0000, the row 2*((pos + b) % 4) of its
//     target bank group (generally elems_per_bank * ...), and the column of its
//     column (by-column mode) or of the previous slot (by-bucket mode).
#include <algorithm>
#include <cstdint>
#include <cstring>
#include <functional>
#include <queue>
#include <utility>
#include <vector>

#include "fq.h"

namespace {

struct Slot {
  uint8_t k;
  uint8_t n;
  uint16_t v;
};

struct Elem {  // one outlier inside a tile
  uint8_t k;
  uint8_t n;
  uint16_t v;
};

fq_status check_params(int32_t K, int32_t N, const fq_tilecoo_params& p) {
  if (K <= 0 || N <= 0) return FQ_ERR_SHAPE;
  if (p.k_tile < 1 || p.k_tile > 256 || p.n_tile < 1 || p.n_tile > 256) return FQ_ERR_FORMAT;
  if (K % p.k_tile != 0 || N % p.n_tile != 0) return FQ_ERR_SHAPE;
  if (p.buckets_per_tile < 1 || p.buckets_per_tile > 1024) return FQ_ERR_FORMAT;
  if (p.group_mode != FQ_GROUP_BY_COLUMN && p.group_mode != FQ_GROUP_BY_BUCKET)
    return FQ_ERR_FORMAT;
  if (p.reorder & ~(FQ_REORDER_COLUMNS | FQ_REORDER_ELEMENTS)) return FQ_ERR_FORMAT;
  if (p.elems_per_bank < 1 || p.n_bank_groups < 1 ||
      int64_t(p.elems_per_bank) * p.n_bank_groups > p.k_tile)
    return FQ_ERR_FORMAT;
  return FQ_OK;
}

// Bank group of a tile-local row index.
inline int bank_group(int k, const fq_tilecoo_params& p) {
  return (k / p.elems_per_bank) % p.n_bank_groups;
}

// Appends `elems` (already in their within-group order) to `out` so that the
// slot at bucket position pos reads bank group (pos + rot) % G when possible.
void append_reordered(const std::vector<Elem>& elems, int rot, const fq_tilecoo_params& p,
                      std::vector<Slot>& out) {
  const int G = p.n_bank_groups;
  std::vector<std::vector<Elem>> queue(G);
  for (const Elem& e : elems) queue[bank_group(e.k, p)].push_back(e);
  std::vector<size_t> head(G, 0);
  for (size_t i = 0; i < elems.size(); ++i) {
    const int target = int((out.size() + rot) % G);
    for (int d = 0; d < G; ++d) {
      const int g = (target + d) % G;
      if (head[g] < queue[g].size()) {
        const Elem& e = queue[g][head[g]++];
        out.push_back({e.k, e.n, e.v});
        break;
      }
    }
  }
}

void pad_to_four(std::vector<Slot>& out, int rot, uint8_t col, const fq_tilecoo_params& p) {
  while (out.size() % 4 != 0) {
    const int gid = int((out.size() + rot) % p.n_bank_groups);
    out.push_back({uint8_t(p.elems_per_bank * gid), col, 0});
  }
}

// Everything the encoder produces, kept until copied out.
struct Encoded {
  std::vector<uint32_t> tile_indptr;
  std::vector<uint16_t> bucket_info;
  std::vector<uint32_t> packed;
  int64_t max_tile_groups = 0;
};

fq_status encode(int32_t K, int32_t N, int64_t nnz, const int32_t* k_idx, const int32_t* n_idx,
                 const uint16_t* val, const fq_tilecoo_params& p, Encoded& enc) {
  const int64_t kt_count = K / p.k_tile;
  const int64_t n_tiles = kt_count * (N / p.n_tile);
  const int B = p.buckets_per_tile;

  // Range checks, then one sort serves both the duplicate check and the
  // grouping by (tile, column, row).
  struct Key {
    uint64_t key;
    uint16_t v;
  };
  std::vector<Key> keys(static_cast<size_t>(nnz));
  for (int64_t i = 0; i < nnz; ++i) {
    const int32_t k = k_idx[i], n = n_idx[i];
    if (k < 0 || k >= K || n < 0 || n >= N) return FQ_ERR_RANGE;
    if ((val[i] & 0x7FFF) == 0) return FQ_ERR_ZERO_VALUE;
    const uint64_t t = uint64_t(n / p.n_tile) * kt_count + uint64_t(k / p.k_tile);
    keys[i].key = (t << 16) | (uint64_t(n % p.n_tile) << 8) | uint64_t(k % p.k_tile);
    keys[i].v = val[i];
  }
  std::sort(keys.begin(), keys.end(), [](const Key& a, const Key& b) { return a.key < b.key; });
  for (size_t i = 1; i < keys.size(); ++i)
    if (keys[i].key == keys[i - 1].key) return FQ_ERR_DUPLICATE;

  enc.tile_indptr.assign(size_t(n_tiles + 1), 0);
  enc.bucket_info.assign(size_t(2 * n_tiles * B), 0);
  enc.packed.clear();
  enc.packed.reserve(size_t(nnz) * 2 + 64);

  std::vector<std::vector<int>> bucket_cols(B);   // column ids, processing order
  std::vector<int> col_start(p.n_tile), col_count(p.n_tile);
  std::vector<int> cols;
  std::vector<Slot> slots;
  std::vector<Elem> elems;
  size_t e = 0;
  for (int64_t t = 0; t < n_tiles; ++t) {
    const size_t e0 = e;
    while (e < keys.size() && (keys[e].key >> 16) == uint64_t(t)) ++e;
    // Column runs inside the tile (entries sorted by column, then row).
    std::fill(col_count.begin(), col_count.end(), 0);
    cols.clear();
    for (size_t i = e0; i < e; ++i) {
      const int c = int((keys[i].key >> 8) & 0xFF);
      if (col_count[c]++ == 0) {
        col_start[c] = int(i);
        cols.push_back(c);
      }
    }
    for (auto& bc : bucket_cols) bc.clear();
    if (p.reorder & FQ_REORDER_COLUMNS) {
      std::vector<int> order(cols);
      std::stable_sort(order.begin(), order.end(), [&](int a, int b) {
        if (col_count[a] != col_count[b]) return col_count[a] > col_count[b];
        return a < b;
      });
      using Load = std::pair<int64_t, int>;  // (nonzeros so far, bucket id)
      std::priority_queue<Load, std::vector<Load>, std::greater<Load>> heap;
      for (int b = 0; b < B; ++b) heap.push({0, b});
      for (int c : order) {
        Load top = heap.top();
        heap.pop();
        bucket_cols[top.second].push_back(c);
        heap.push({top.first + col_count[c], top.second});
      }
    } else {
      for (int c : cols) bucket_cols[int64_t(c) * B / p.n_tile].push_back(c);
    }

    const size_t tile_first = enc.packed.size() / 4;
    enc.tile_indptr[t] = uint32_t(tile_first);
    for (int b = 0; b < B; ++b) {
      const int rot = b % p.n_bank_groups;
      slots.clear();
      if (p.group_mode == FQ_GROUP_BY_COLUMN) {
        for (int c : bucket_cols[b]) {
          elems.clear();
          for (int i = 0; i < col_count[c]; ++i) {
            const Key& kk = keys[size_t(col_start[c] + i)];
            elems.push_back({uint8_t(kk.key & 0xFF), uint8_t(c), kk.v});
          }
          if (p.reorder & FQ_REORDER_ELEMENTS) {
            append_reordered(elems, rot, p, slots);
          } else {
            for (const Elem& x : elems) slots.push_back({x.k, x.n, x.v});
          }
          pad_to_four(slots, rot, uint8_t(c), p);
        }
      } else {
        elems.clear();
        for (int c : bucket_cols[b])
          for (int i = 0; i < col_count[c]; ++i) {
            const Key& kk = keys[size_t(col_start[c] + i)];
            elems.push_back({uint8_t(kk.key & 0xFF), uint8_t(c), kk.v});
          }
        if (p.reorder & FQ_REORDER_ELEMENTS) {
          // Within a bank-group queue: by row, then by the column's position
          // in the bucket.  Elements arrive grouped by column in bucket order,
          // so a stable sort by row keeps that secondary order.
          std::stable_sort(elems.begin(), elems.end(),
                           [](const Elem& a, const Elem& b) { return a.k < b.k; });
          append_reordered(elems, rot, p, slots);
        } else {
          for (const Elem& x : elems) slots.push_back({x.k, x.n, x.v});
        }
        if (!slots.empty()) pad_to_four(slots, rot, slots.back().n, p);
      }
      const size_t offset = enc.packed.size() / 4 - tile_first;
      const size_t count = slots.size() / 4;
      if (offset > 0xFFFF || count > 0xFFFF) return FQ_ERR_FORMAT;
      enc.bucket_info[size_t(2 * (t * B + b))] = uint16_t(offset);
      enc.bucket_info[size_t(2 * (t * B + b) + 1)] = uint16_t(count);
      for (size_t g = 0; g < count; ++g) {
        const Slot* s = &slots[4 * g];
        enc.packed.push_back(uint32_t(s[0].k) | uint32_t(s[1].k) << 8 | uint32_t(s[2].k) << 16 |
                             uint32_t(s[3].k) << 24);
        enc.packed.push_back(uint32_t(s[0].n) | uint32_t(s[1].n) << 8 | uint32_t(s[2].n) << 16 |
                             uint32_t(s[3].n) << 24);
        enc.packed.push_back(uint32_t(s[0].v) | uint32_t(s[1].v) << 16);
        enc.packed.push_back(uint32_t(s[2].v) | uint32_t(s[3].v) << 16);
      }
    }
    enc.max_tile_groups =
        std::max<int64_t>(enc.max_tile_groups, int64_t(enc.packed.size() / 4 - tile_first));
  }
  enc.tile_indptr[size_t(n_tiles)] = uint32_t(enc.packed.size() / 4);
  if (enc.packed.size() / 4 > 0xFFFFFFFFull) return FQ_ERR_FORMAT;
  return FQ_OK;
}

void fill_sizes(const fq_tilecoo_params& p, int64_t n_tiles, int64_t n_groups, int64_t nnz,
                int64_t max_tile_groups, fq_tilecoo_sizes* s) {
  s->n_tiles = n_tiles;
  s->n_buckets = n_tiles * p.buckets_per_tile;
  s->n_groups = n_groups;
  s->nnz = nnz;
  s->n_pad = 4 * n_groups - nnz;
  s->bytes = 4 * (n_tiles + 1) + 4 * s->n_buckets + 16 * n_groups;
  s->max_tile_groups = max_tile_groups;
}

}  // namespace

extern "C" {

fq_tilecoo_params fq_default_tilecoo_params(void) {
  fq_tilecoo_params p;
  p.k_tile = 128;
  p.n_tile = 64;
  p.buckets_per_tile = 1;
  p.group_mode = FQ_GROUP_BY_BUCKET;
  p.reorder = FQ_REORDER_COLUMNS | FQ_REORDER_ELEMENTS;
  p.elems_per_bank = 2;
  p.n_bank_groups = 4;
  return p;
}

fq_status fq_pack_tile_coo(int32_t K, int32_t N, int64_t nnz, const int32_t* k_idx,
                           const int32_t* n_idx, const uint16_t* val,
                           const fq_tilecoo_params* pp, fq_tilecoo_sizes* sizes,
                           uint32_t* tile_indptr, uint16_t* bucket_info, uint32_t* packed) {
  try {
    const fq_tilecoo_params p = pp ? *pp : fq_default_tilecoo_params();
    if (!sizes) return FQ_ERR_NULL;
    if (nnz < 0) return FQ_ERR_SHAPE;
    if (nnz > 0 && (!k_idx || !n_idx || !val)) return FQ_ERR_NULL;
    const bool size_only = !tile_indptr && !bucket_info && !packed;
    if (!size_only && (!tile_indptr || !bucket_info || !packed)) return FQ_ERR_NULL;
    fq_status st = check_params(K, N, p);
    if (st != FQ_OK) return st;
    Encoded enc;
    st = encode(K, N, nnz, k_idx, n_idx, val, p, enc);
    if (st != FQ_OK) return st;
    const int64_t n_tiles = int64_t(enc.tile_indptr.size()) - 1;
    const int64_t n_groups = int64_t(enc.packed.size() / 4);
    fill_sizes(p, n_tiles, n_groups, nnz, enc.max_tile_groups, sizes);
    if (!size_only) {
      std::memcpy(tile_indptr, enc.tile_indptr.data(), enc.tile_indptr.size() * 4);
      std::memcpy(bucket_info, enc.bucket_info.data(), enc.bucket_info.size() * 2);
      if (!enc.packed.empty()) std::memcpy(packed, enc.packed.data(), enc.packed.size() * 4);
    }
    return FQ_OK;
  } catch (...) {
    return FQ_ERR_FORMAT;
  }
}

fq_status fq_validate_tile_coo(int32_t K, int32_t N, const fq_tilecoo_params* pp,
                               int64_t n_groups, const uint32_t* tile_indptr,
                               const uint16_t* bucket_info, const uint32_t* packed) {
  try {
    if (!pp || !tile_indptr || !bucket_info || (n_groups > 0 && !packed)) return FQ_ERR_NULL;
    const fq_tilecoo_params& p = *pp;
    fq_status st = check_params(K, N, p);
    if (st != FQ_OK) return st;
    if (n_groups < 0) return FQ_ERR_FORMAT;
    const int64_t n_tiles = int64_t(K / p.k_tile) * (N / p.n_tile);
    const int B = p.buckets_per_tile;
    if (tile_indptr[0] != 0 || int64_t(tile_indptr[n_tiles]) != n_groups) return FQ_ERR_FORMAT;
    std::vector<int> owner(size_t(p.n_tile));
    std::vector<uint8_t> seen(size_t(p.k_tile) * p.n_tile, 0);
    std::vector<int> touched;
    for (int64_t t = 0; t < n_tiles; ++t) {
      const int64_t g0 = tile_indptr[t], g1 = tile_indptr[t + 1];
      if (g1 < g0) return FQ_ERR_FORMAT;
      std::fill(owner.begin(), owner.end(), -1);
      int64_t expect = 0;
      for (int b = 0; b < B; ++b) {
        const int64_t off = bucket_info[size_t(2 * (t * B + b))];
        const int64_t cnt = bucket_info[size_t(2 * (t * B + b) + 1)];
        if (off != expect) return FQ_ERR_FORMAT;
        expect += cnt;
        if (g0 + expect > g1) return FQ_ERR_FORMAT;
        for (int64_t g = g0 + off; g < g0 + off + cnt; ++g) {
          const uint32_t* w = packed + 4 * g;
          int first_col = -1;
          for (int j = 0; j < 4; ++j) {
            const int k = int((w[0] >> (8 * j)) & 0xFF);
            const int n = int((w[1] >> (8 * j)) & 0xFF);
            const uint16_t v = uint16_t((w[2 + j / 2] >> (16 * (j % 2))) & 0xFFFF);
            if (k >= p.k_tile || n >= p.n_tile) return FQ_ERR_FORMAT;
            if (p.group_mode == FQ_GROUP_BY_COLUMN) {
              if (first_col < 0) first_col = n;
              if (n != first_col) return FQ_ERR_FORMAT;
            }
            if (v == 0) continue;
            if ((v & 0x7FFF) == 0) return FQ_ERR_FORMAT;
            if (owner[size_t(n)] < 0) owner[size_t(n)] = b;
            if (owner[size_t(n)] != b) return FQ_ERR_FORMAT;
            const size_t pos = size_t(k) * p.n_tile + size_t(n);
            if (seen[pos]) return FQ_ERR_FORMAT;
            seen[pos] = 1;
            touched.push_back(int(pos));
          }
        }
      }
      if (g0 + expect != g1) return FQ_ERR_FORMAT;
      for (int pos : touched) seen[size_t(pos)] = 0;
      touched.clear();
    }
    return FQ_OK;
  } catch (...) {
    return FQ_ERR_FORMAT;
  }
}

fq_status fq_unpack_tile_coo(int32_t K, int32_t N, const fq_tilecoo_params* pp, int64_t n_groups,
                             const uint32_t* tile_indptr, const uint16_t* bucket_info,
                             const uint32_t* packed, int64_t* nnz_out, int32_t* k_idx,
                             int32_t* n_idx, uint16_t* val) {
  try {
    if (!nnz_out) return FQ_ERR_NULL;
    fq_status st = fq_validate_tile_coo(K, N, pp, n_groups, tile_indptr, bucket_info, packed);
    if (st != FQ_OK) return st;
    const fq_tilecoo_params& p = *pp;
    const bool count_only = !k_idx && !n_idx && !val;
    if (!count_only && (!k_idx || !n_idx || !val)) return FQ_ERR_NULL;
    const int64_t kt_count = K / p.k_tile;
    const int64_t n_tiles = kt_count * (N / p.n_tile);
    struct Trip {
      int64_t pos;
      uint16_t v;
    };
    std::vector<Trip> out;
    for (int64_t t = 0; t < n_tiles; ++t) {
      const int64_t k0 = (t % kt_count) * p.k_tile;
      const int64_t n0 = (t / kt_count) * p.n_tile;
      for (int b = 0; b < p.buckets_per_tile; ++b) {
        const int64_t off = bucket_info[size_t(2 * (t * p.buckets_per_tile + b))];
        const int64_t cnt = bucket_info[size_t(2 * (t * p.buckets_per_tile + b) + 1)];
        for (int64_t g = tile_indptr[t] + off; g < tile_indptr[t] + off + cnt; ++g) {
          const uint32_t* w = packed + 4 * g;
          for (int j = 0; j < 4; ++j) {
            const uint16_t v = uint16_t((w[2 + j / 2] >> (16 * (j % 2))) & 0xFFFF);
            if (v == 0) continue;
            const int64_t k = k0 + ((w[0] >> (8 * j)) & 0xFF);
            const int64_t n = n0 + ((w[1] >> (8 * j)) & 0xFF);
            out.push_back({k * N + n, v});
          }
        }
      }
    }
    if (!count_only && int64_t(out.size()) != *nnz_out) return FQ_ERR_SHAPE;
    *nnz_out = int64_t(out.size());
    if (count_only) return FQ_OK;
    std::sort(out.begin(), out.end(), [](const Trip& a, const Trip& b) { return a.pos < b.pos; });
    for (size_t i = 0; i < out.size(); ++i) {
      k_idx[i] = int32_t(out[i].pos / N);
      n_idx[i] = int32_t(out[i].pos % N);
      val[i] = out[i].v;
    }
    return FQ_OK;
  } catch (...) {
    return FQ_ERR_FORMAT;
  }
}

}  // extern "C"
