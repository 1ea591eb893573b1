// Offline outlier-aware INT4 quantiser (host).  Splits a dense weight matrix
// into the low-bit part W_Q (per-group affine INT4, eq. 2 and eq. 3 of the
// paper) and the bf16 outlier part W_O (the highest-magnitude weights, Sec. 2.2),
// and optionally stores original weights in the Tile-COO padding slots
// (Sec. 3.2.1: padding slots may hold original weight values).
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <numeric>
#include <unordered_set>
#include <vector>

#include "fq.h"

namespace {

constexpr int kLevels = 15;   // 2^4 - 1

// Smallest fp16 value >= s, for 0 < s <= 65504; returns its bit pattern.
uint16_t f16_bits_at_least(double s) {
  if (s < std::ldexp(1.0, -14)) {                       // subnormal range, unit 2^-24
    const double f = std::ceil(std::ldexp(s, 24));      // 1..1024 (1024 = smallest normal)
    return uint16_t(f);
  }
  int e = 0;
  std::frexp(s, &e);                                    // s = m 2^e, m in [0.5, 1)
  int E = e - 1;                                        // s in [2^E, 2^(E+1))
  double f = std::ceil((std::ldexp(s, -E) - 1.0) * 1024.0);
  if (f >= 1024.0) {
    f = 0.0;
    ++E;
  }
  return uint16_t(((E + 15) << 10) | int(f));
}

double f16_value(uint16_t h) {
  const int e = (h >> 10) & 31, f = h & 1023;
  const double mag = e == 0 ? std::ldexp(double(f), -24) : std::ldexp(1.0 + f / 1024.0, e - 15);
  return (h & 0x8000) ? -mag : mag;
}

// fp32 -> bf16 bits, round to nearest, ties to even (finite input).
uint16_t bf16_bits(float w) {
  uint32_t u;
  std::memcpy(&u, &w, 4);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return uint16_t(u >> 16);
}

// Round to nearest integer, ties to even.
double rne(double x) { return std::nearbyint(x); }

struct GroupQuant {
  uint16_t s_bits;
  double s;
  int z;
};

// eq. 2 on one group's non-outlier weights: the range is widened to hold 0
// so the zero-point fits the unsigned code range, the scale is stored as the
// smallest fp16 not below (w_max - w_min) / 15, and an all-zero group gets
// scale 1 and zero-point 0.
GroupQuant quantise_group(double w_min, double w_max) {
  w_min = std::min(w_min, 0.0);
  w_max = std::max(w_max, 0.0);
  GroupQuant g;
  const double s = (w_max - w_min) / kLevels;
  if (s == 0.0) {
    g.s_bits = 0x3C00;   // 1.0
    g.s = 1.0;
    g.z = 0;
    return g;
  }
  g.s_bits = f16_bits_at_least(s);
  g.s = f16_value(g.s_bits);
  g.z = int(std::min(double(kLevels), std::max(0.0, rne(-w_min / g.s))));
  return g;
}

int code_of(double w, const GroupQuant& g) {
  return int(std::min(double(kLevels), std::max(0.0, rne(w / g.s) + g.z)));
}

}  // namespace

extern "C" {

fq_status fq_quantize_outlier_aware(int32_t K, int32_t N, const float* W, int32_t group_size,
                                    double outlier_frac, int64_t* nnz_out, uint32_t* Wq,
                                    uint16_t* scales, uint32_t* zeros, int32_t* k_idx,
                                    int32_t* n_idx, uint16_t* val) {
  if (!W || !nnz_out) return FQ_ERR_NULL;
  if (K <= 0 || N <= 0 || group_size <= 0 || K % group_size || K % 8 || N % 8) return FQ_ERR_SHAPE;
  if (!(outlier_frac >= 0.0 && outlier_frac <= 1.0)) return FQ_ERR_RANGE;
  const int64_t total = int64_t(K) * N;
  for (int64_t i = 0; i < total; ++i)
    if (!std::isfinite(W[i])) return FQ_ERR_RANGE;

  // Outliers: the round(frac K N) largest |w| (ties to the lower row-major
  // index) among weights whose bf16 value is nonzero, since bf16 0 marks a
  // padding slot.
  std::vector<int64_t> cand;
  cand.reserve(size_t(total));
  for (int64_t i = 0; i < total; ++i)
    if ((bf16_bits(W[i]) & 0x7FFFu) != 0u) cand.push_back(i);
  const int64_t want = std::min<int64_t>(int64_t(rne(outlier_frac * double(total))),
                                         int64_t(cand.size()));
  auto before = [W](int64_t a, int64_t b) {
    const float fa = std::fabs(W[a]), fb = std::fabs(W[b]);
    return fa != fb ? fa > fb : a < b;
  };
  if (want < int64_t(cand.size()))
    std::nth_element(cand.begin(), cand.begin() + want, cand.end(), before);
  cand.resize(size_t(want));
  std::sort(cand.begin(), cand.end());   // row-major order = sorted by (k, n)
  *nnz_out = want;
  const bool sizes_only = !Wq && !scales && !zeros && !k_idx && !n_idx && !val;
  if (sizes_only) return FQ_OK;
  if (!Wq || !scales || !zeros || (want > 0 && (!k_idx || !n_idx || !val))) return FQ_ERR_NULL;

  std::vector<uint8_t> is_out(size_t(total), 0);
  for (int64_t i = 0; i < want; ++i) {
    const int64_t p = cand[size_t(i)];
    is_out[size_t(p)] = 1;
    k_idx[i] = int32_t(p / N);
    n_idx[i] = int32_t(p % N);
    val[i] = bf16_bits(W[p]);
  }

  const int32_t G = K / group_size;
  std::memset(Wq, 0, size_t(K / 8) * N * 4);
  std::memset(zeros, 0, size_t(G) * (N / 8) * 4);
  for (int32_t g = 0; g < G; ++g) {
    for (int32_t n = 0; n < N; ++n) {
      double lo = 0.0, hi = 0.0;
      for (int32_t k = g * group_size; k < (g + 1) * group_size; ++k) {
        const int64_t p = int64_t(k) * N + n;
        if (is_out[size_t(p)]) continue;
        lo = std::min(lo, double(W[p]));
        hi = std::max(hi, double(W[p]));
      }
      const GroupQuant gq = quantise_group(lo, hi);
      scales[size_t(g) * N + n] = gq.s_bits;
      zeros[size_t(g) * (N / 8) + n / 8] |= uint32_t(gq.z) << (4 * (n % 8));
      for (int32_t k = g * group_size; k < (g + 1) * group_size; ++k) {
        const int64_t p = int64_t(k) * N + n;
        // the dense part contributes nothing where an outlier sits
        const int q = is_out[size_t(p)] ? gq.z : code_of(double(W[p]), gq);
        Wq[size_t(k / 8) * N + n] |= uint32_t(q) << (4 * (k % 8));
      }
    }
  }
  return FQ_OK;
}

fq_status fq_fill_padding_slots(int32_t K, int32_t N, const float* W, int32_t group_size,
                                const fq_tilecoo_params* p, int64_t n_groups,
                                const uint32_t* tile_indptr, const uint16_t* bucket_info,
                                uint32_t* packed, uint32_t* Wq, const uint32_t* zeros,
                                int64_t* n_filled) {
  if (!W || !p || !tile_indptr || !bucket_info || !Wq || !zeros || !n_filled) return FQ_ERR_NULL;
  if (n_groups > 0 && !packed) return FQ_ERR_NULL;
  if (group_size <= 0 || K % group_size) return FQ_ERR_SHAPE;
  fq_status st = fq_validate_tile_coo(K, N, p, n_groups, tile_indptr, bucket_info, packed);
  if (st != FQ_OK) return st;
  *n_filled = 0;
  const int32_t kt_count = K / p->k_tile;
  const int64_t n_tiles = int64_t(kt_count) * (N / p->n_tile);
  for (int64_t t = 0; t < n_tiles; ++t) {
    const int64_t kb = (t % kt_count) * p->k_tile, nb = (t / kt_count) * p->n_tile;
    const uint32_t g0 = tile_indptr[t], g1 = tile_indptr[t + 1];
    // positions already holding a real value in this tile
    std::unordered_set<uint32_t> used;
    for (uint32_t g = g0; g < g1; ++g) {
      const uint32_t* q = packed + 4 * size_t(g);
      for (int j = 0; j < 4; ++j) {
        const uint16_t v = uint16_t((q[2 + j / 2] >> (16 * (j & 1))) & 0xFFFFu);
        if (v != 0) used.insert(((q[0] >> (8 * j)) & 0xFFu) << 8 | ((q[1] >> (8 * j)) & 0xFFu));
      }
    }
    for (uint32_t g = g0; g < g1; ++g) {
      uint32_t* q = packed + 4 * size_t(g);
      for (int j = 0; j < 4; ++j) {
        const uint32_t sh = 16 * (j & 1);
        if (((q[2 + j / 2] >> sh) & 0xFFFFu) != 0) continue;
        const uint32_t kl = (q[0] >> (8 * j)) & 0xFFu, nl = (q[1] >> (8 * j)) & 0xFFu;
        const uint32_t key = kl << 8 | nl;
        if (used.count(key)) continue;
        const int64_t k = kb + kl, n = nb + nl;
        const uint16_t v = bf16_bits(W[k * N + n]);
        if ((v & 0x7FFFu) == 0) continue;
        used.insert(key);
        q[2 + j / 2] = (q[2 + j / 2] & ~(0xFFFFu << sh)) | (uint32_t(v) << sh);
        // the slot now carries the weight exactly: its code becomes the
        // group's zero-point so the dense part adds nothing there
        const uint32_t z = (zeros[size_t(k / group_size) * (N / 8) + n / 8] >> (4 * (n % 8))) & 15u;
        uint32_t& word = Wq[size_t(k / 8) * N + n];
        word = (word & ~(15u << (4 * (k % 8)))) | (z << (4 * (k % 8)));
        ++*n_filled;
      }
    }
  }
  return FQ_OK;
}

}  // extern "C"
