// C ABI: argument validation and dispatch to the HIP launchers.  Every check
// runs on the host before anything is enqueued.
#include <cstdint>

#include "fq.h"
#include "internal.hpp"

static_assert(FQ_NOALLOC_SCRATCH_BYTES == fqi::kScratchBytes, "static scratch size in fq.h");

namespace {

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

fq_status check_problem(const fq_problem* pr) {
  if (!pr) return FQ_ERR_NULL;
  if (pr->M < 1 || pr->K < 1 || pr->N < 1 || pr->split_k < 0) return FQ_ERR_SHAPE;
  if (pr->K % fqi::kTileK != 0 || pr->N % fqi::kTileN != 0) return FQ_ERR_SHAPE;
  if (pr->group_size != fqi::kTileK) return FQ_ERR_UNSUPPORTED;
  if (pr->M > fqi::kMaxM) return FQ_ERR_UNSUPPORTED;
  if (pr->y_dtype != FQ_Y_BF16 && pr->y_dtype != FQ_Y_F32) return FQ_ERR_UNSUPPORTED;
  if (pr->flags & ~(FQ_SPARSE_MASK | FQ_SCHED_STREAM_K | FQ_FOUR_WAVES | FQ_STRIP_32 | FQ_STRIP_64 |
                    FQ_SPARSE_WAVES | FQ_DENSE_VALU))
    return FQ_ERR_UNSUPPORTED;
  if ((pr->flags & FQ_DENSE_VALU) &&
      (pr->M != 1 || (pr->flags & (FQ_SCHED_STREAM_K | FQ_SPARSE_WAVES)) ||
       (pr->flags & FQ_SPARSE_MASK) == FQ_SPARSE_GATHER))
    return FQ_ERR_UNSUPPORTED;
  const int mapping = pr->flags & FQ_SPARSE_MASK;
  if ((pr->flags & FQ_STRIP_32) &&
      ((pr->flags & (FQ_STRIP_64 | FQ_SCHED_STREAM_K)) || mapping == FQ_SPARSE_GATHER))
    return FQ_ERR_UNSUPPORTED;
  if (mapping > FQ_SPARSE_MFMA) return FQ_ERR_UNSUPPORTED;
  if (mapping == FQ_SPARSE_GATHER && pr->M > fqi::kGatherLimitM) return FQ_ERR_UNSUPPORTED;
  return FQ_OK;
}

fq_status check_dense_ptrs(const uint16_t* X, const uint32_t* Wq, const uint16_t* scales,
                           const uint32_t* zeros, const void* Y) {
  if (!X || !Wq || !scales || !zeros || !Y) return FQ_ERR_NULL;
  if (!aligned(X, 16) || !aligned(Wq, 16) || !aligned(scales, 8) || !aligned(zeros, 4) ||
      !aligned(Y, 16))
    return FQ_ERR_ALIGN;
  return FQ_OK;
}

fq_status check_tc(const fq_problem* pr, const fq_tilecoo_dev* tc) {
  if (!tc) return FQ_ERR_NULL;
  const fq_tilecoo_params& p = tc->params;
  if (p.k_tile != fqi::kTileK || p.n_tile != fqi::kTileN) return FQ_ERR_UNSUPPORTED;
  if (p.buckets_per_tile < 1 || p.buckets_per_tile > fqi::kMaxBuckets) return FQ_ERR_UNSUPPORTED;
  if (p.group_mode != FQ_GROUP_BY_COLUMN && p.group_mode != FQ_GROUP_BY_BUCKET) return FQ_ERR_FORMAT;
  if (tc->n_groups < 0 || tc->max_tile_groups < 0) return FQ_ERR_FORMAT;
  if (tc->n_groups >= (int64_t(1) << 27)) return FQ_ERR_UNSUPPORTED;   // 16-byte groups < 2^31 B
  if (!tc->tile_indptr || !tc->bucket_info || (tc->n_groups > 0 && !tc->packed)) return FQ_ERR_NULL;
  if (!aligned(tc->tile_indptr, 4) || !aligned(tc->bucket_info, 4) || !aligned(tc->packed, 16))
    return FQ_ERR_ALIGN;
  (void)pr;
  return FQ_OK;
}

int plan_opts(const fq_problem* pr);

// Sparse mapping for make_plan: the caller's, else -1 (by M) -- except that
// groups whose slots may lie in different columns (by-bucket grouping) always
// take the MFMA mapping, which scatters every slot on its own; the gather
// mapping is built around single-column groups.
int plan_mode(const fq_problem* pr, int32_t group_mode) {
  const int mapping = pr->flags & FQ_SPARSE_MASK;
  if (mapping == FQ_SPARSE_GATHER) return 0;
  if (mapping == FQ_SPARSE_MFMA || group_mode == FQ_GROUP_BY_BUCKET || (pr->flags & FQ_DENSE_VALU))
    return 1;
  return -1;
}

bool plan_for(const fq_problem* pr, const fq_tilecoo_dev* tc, bool dense, bool sparse,
              fqi::Plan* plan) {
  const int mode = plan_mode(pr, sparse ? tc->params.group_mode : FQ_GROUP_BY_COLUMN);
  return fqi::make_plan(pr->M, pr->K, pr->N, pr->split_k, dense, sparse,
                        sparse ? tc->params.buckets_per_tile : 0,
                        sparse ? tc->max_tile_groups : 0, plan, mode, plan_opts(pr));
}

fq_status run(const fq_problem* pr, const uint16_t* X, const uint32_t* Wq,
              const uint16_t* scales, const uint32_t* zeros, const fq_tilecoo_dev* tc, void* Y,
              void* workspace, size_t workspace_bytes, void* stream, bool dense, bool sparse,
              const float* y_addend) {
  fqi::Plan plan;
  if (!plan_for(pr, tc, dense, sparse, &plan)) return FQ_ERR_UNSUPPORTED;
  if (!workspace) return FQ_ERR_WORKSPACE;
  if (workspace_bytes < plan.ws_bytes || !aligned(workspace, 256)) return FQ_ERR_WORKSPACE;
  fqi::MatmulPtrs p{};
  p.X = X;
  p.Wq = Wq;
  p.scales = scales;
  p.zeros = zeros;
  if (sparse) {
    p.tile_indptr = tc->tile_indptr;
    p.bucket_info = tc->bucket_info;
    p.packed = tc->packed;
    p.n_groups = tc->n_groups;
  }
  p.y_addend = y_addend;
  p.Y = Y;
  p.y_f32 = pr->y_dtype == FQ_Y_F32;
  p.workspace = workspace;
  return fqi::launch_matmul(plan, p, dense, sparse, stream) == 0 ? FQ_OK : FQ_ERR_HIP;
}

size_t align256(size_t x) { return (x + 255) / 256 * 256; }

int plan_opts(const fq_problem* pr) {
  return ((pr->flags & FQ_SCHED_STREAM_K) ? fqi::kOptStreamK : 0) |
         ((pr->flags & FQ_FOUR_WAVES) ? fqi::kOptFourWaves : 0) |
         ((pr->flags & FQ_STRIP_32) ? fqi::kOptStrip32 : 0) |
         ((pr->flags & FQ_STRIP_64) ? fqi::kOptStrip64 : 0) |
         ((pr->flags & FQ_SPARSE_WAVES) ? fqi::kOptSparseWaves : 0) |
         ((pr->flags & FQ_DENSE_VALU) ? fqi::kOptDenseValu : 0);
}

}  // namespace

extern "C" {

const char* fq_status_string(fq_status s) {
  switch (s) {
    case FQ_OK: return "ok";
    case FQ_ERR_NULL: return "required pointer is NULL";
    case FQ_ERR_SHAPE: return "invalid or indivisible shape";
    case FQ_ERR_RANGE: return "COO index out of range";
    case FQ_ERR_DUPLICATE: return "duplicate COO position";
    case FQ_ERR_ZERO_VALUE: return "zero-valued outlier";
    case FQ_ERR_FORMAT: return "inconsistent Tile-COO arrays or parameters";
    case FQ_ERR_UNSUPPORTED: return "unsupported configuration";
    case FQ_ERR_WORKSPACE: return "workspace missing, misaligned or too small";
    case FQ_ERR_HIP: return "HIP runtime error at launch";
    case FQ_ERR_ALIGN: return "device pointer misaligned";
    case FQ_ERR_SCRATCH_LIMIT: return "problem needs more scratch than the static maximum";
  }
  return "unknown status";
}

fq_status fq_launch_config(const fq_problem* pr, int32_t buckets_per_tile, int32_t group_mode,
                           int32_t cfg[10]) {
  if (!cfg) return FQ_ERR_NULL;
  fq_status st = check_problem(pr);
  if (st != FQ_OK) return st;
  if (group_mode != FQ_GROUP_BY_COLUMN && group_mode != FQ_GROUP_BY_BUCKET) return FQ_ERR_FORMAT;
  const int mode = plan_mode(pr, group_mode);
  fqi::Plan pl;
  if (!fqi::make_plan(pr->M, pr->K, pr->N, pr->split_k, true, true, buckets_per_tile, 0, &pl, mode,
                      plan_opts(pr)))
    return FQ_ERR_UNSUPPORTED;
  cfg[0] = 16 * pl.NCB;
  cfg[1] = pl.S;
  cfg[2] = pl.NW;
  cfg[3] = pl.NWS;
  cfg[4] = pl.MODE == 0 ? FQ_SPARSE_GATHER : FQ_SPARSE_MFMA;
  cfg[5] = pl.G * pl.n_slabs;
  cfg[6] = pl.stream;
  cfg[7] = int32_t(pl.lds_bytes);
  cfg[8] = pl.XS;
  cfg[9] = pl.BK;
  return FQ_OK;
}

fq_status fq_workspace_bytes(const fq_problem* pr, size_t* bytes) {
  if (!bytes) return FQ_ERR_NULL;
  fq_status st = check_problem(pr);
  if (st != FQ_OK) return st;
  // The split, and with it the partial-sum area, depends on the kernel the
  // call launches: size for the largest of dense-only and both mappings.
  fqi::Plan pl;
  size_t need = 0;
  bool any = false;
  for (int mode = -1; mode <= 1; ++mode) {
    for (int sparse = 0; sparse <= 1; ++sparse) {
      if (fqi::make_plan(pr->M, pr->K, pr->N, pr->split_k, true, sparse != 0, 1, 0, &pl, mode,
                         plan_opts(pr))) {
        any = true;
        need = pl.ws_bytes > need ? pl.ws_bytes : need;
      }
    }
  }
  if (!any) return FQ_ERR_UNSUPPORTED;
  *bytes = need;
  return FQ_OK;
}

fq_status fq_workspace_bytes_unfused(const fq_problem* pr, size_t* bytes) {
  size_t base = 0;
  fq_status st = fq_workspace_bytes(pr, &base);
  if (st != FQ_OK) return st;
  *bytes = align256(base) + align256(size_t(pr->M) * size_t(pr->N) * 4);
  return FQ_OK;
}

fq_status fq_w4a16_outlier_matmul(const fq_problem* pr, const uint16_t* X, const uint32_t* Wq,
                                  const uint16_t* scales, const uint32_t* zeros,
                                  const fq_tilecoo_dev* tc, void* Y, void* workspace,
                                  size_t workspace_bytes, void* stream) {
  fq_status st = check_problem(pr);
  if (st == FQ_OK) st = check_dense_ptrs(X, Wq, scales, zeros, Y);
  if (st == FQ_OK) st = check_tc(pr, tc);
  if (st != FQ_OK) return st;
  return run(pr, X, Wq, scales, zeros, tc, Y, workspace, workspace_bytes, stream, true, true,
             nullptr);
}

fq_status fq_w4a16_outlier_matmul_noalloc(const fq_problem* pr, const uint16_t* X,
                                          const uint32_t* Wq, const uint16_t* scales,
                                          const uint32_t* zeros, const fq_tilecoo_dev* tc,
                                          void* Y, void* stream) {
  fq_status st = check_problem(pr);
  if (st == FQ_OK) st = check_dense_ptrs(X, Wq, scales, zeros, Y);
  if (st == FQ_OK) st = check_tc(pr, tc);
  if (st != FQ_OK) return st;
  // the same plan the workspace entry point makes; its workspace must fit
  // the static scratch (checked before the device is touched)
  fqi::Plan plan;
  if (!plan_for(pr, tc, true, true, &plan)) return FQ_ERR_UNSUPPORTED;
  if (plan.ws_bytes > fqi::kScratchBytes) return FQ_ERR_SCRATCH_LIMIT;
  void* scratch = nullptr;
  if (fqi::scratch_for_current_device(&scratch, stream) != 0) return FQ_ERR_HIP;
  return run(pr, X, Wq, scales, zeros, tc, Y, scratch, fqi::kScratchBytes, stream, true, true,
             nullptr);
}

fq_status fq_w4a16_matmul(const fq_problem* pr, const uint16_t* X, const uint32_t* Wq,
                          const uint16_t* scales, const uint32_t* zeros, void* Y,
                          void* workspace, size_t workspace_bytes, void* stream) {
  fq_status st = check_problem(pr);
  if (st == FQ_OK) st = check_dense_ptrs(X, Wq, scales, zeros, Y);
  if (st != FQ_OK) return st;
  return run(pr, X, Wq, scales, zeros, nullptr, Y, workspace, workspace_bytes, stream, true,
             false, nullptr);
}

fq_status fq_w4a16_outlier_matmul_unfused(const fq_problem* pr, const uint16_t* X,
                                          const uint32_t* Wq, const uint16_t* scales,
                                          const uint32_t* zeros, const fq_tilecoo_dev* tc,
                                          void* Y, void* workspace, size_t workspace_bytes,
                                          void* stream) {
  fq_status st = check_problem(pr);
  if (st == FQ_OK) st = check_dense_ptrs(X, Wq, scales, zeros, Y);
  if (st == FQ_OK) st = check_tc(pr, tc);
  if (st != FQ_OK) return st;
  size_t need = 0, base = 0;
  if ((st = fq_workspace_bytes_unfused(pr, &need)) != FQ_OK) return st;
  if ((st = fq_workspace_bytes(pr, &base)) != FQ_OK) return st;
  if (!workspace || workspace_bytes < need || !aligned(workspace, 256)) return FQ_ERR_WORKSPACE;
  float* ydense = reinterpret_cast<float*>(static_cast<char*>(workspace) + align256(base));
  // Kernel 1: dense-only W4A16, fp32 result into the workspace.
  fq_problem p1 = *pr;
  p1.y_dtype = FQ_Y_F32;
  st = run(&p1, X, Wq, scales, zeros, nullptr, ydense, workspace, base, stream, true, false,
           nullptr);
  if (st != FQ_OK) return st;
  // Kernel 2: Tile-COO SpMM re-reading X, adding the dense result.
  return run(pr, X, Wq, scales, zeros, tc, Y, workspace, base, stream, false, true, ydense);
}

fq_status fq_debug_decode_tile_coo(const fq_tilecoo_dev* tc, int32_t K, int32_t N,
                                   int32_t* k_out, int32_t* n_out, uint16_t* v_out,
                                   void* stream) {
  if (!tc) return FQ_ERR_NULL;
  const fq_tilecoo_params& p = tc->params;
  if (p.k_tile < 1 || p.k_tile > 256 || p.n_tile < 1 || p.n_tile > 256) return FQ_ERR_FORMAT;
  if (K < 1 || N < 1 || K % p.k_tile || N % p.n_tile) return FQ_ERR_SHAPE;
  if (tc->n_groups < 0) return FQ_ERR_FORMAT;
  if (tc->n_groups == 0) return FQ_OK;
  if (!tc->tile_indptr || !tc->packed || !k_out || !n_out || !v_out) return FQ_ERR_NULL;
  if (!aligned(tc->packed, 16) || !aligned(tc->tile_indptr, 4) || !aligned(k_out, 4) ||
      !aligned(n_out, 4) || !aligned(v_out, 2))
    return FQ_ERR_ALIGN;
  const int kt_count = K / p.k_tile;
  const int64_t n_tiles = int64_t(kt_count) * (N / p.n_tile);
  return fqi::launch_decode(tc->tile_indptr, n_tiles, tc->packed, tc->n_groups, kt_count,
                            p.k_tile, p.n_tile, k_out, n_out, v_out, stream) == 0
             ? FQ_OK
             : FQ_ERR_HIP;
}

}  // extern "C"
