// Launch plan shared by the planner (gts_kernels.hip) and the translation
// units that instantiate the SHAP kernels (gts_shap_f32.hip and friends).
// Not part of the public ABI.
#pragma once

#include <cstddef>
#include <cstdint>

#include "gts_internal.h"

namespace gts {

// Longest path (features) with fully unrolled per-path code.  Longer paths
// run the runtime-loop code, in fp64, which keeps its per-path arrays in
// per-lane private memory; only the long-path kernel variants contain it.
constexpr int kMaxUnrolledShap = 12;
constexpr int kMaxUnrolledInter = 8;
// SHAP paths of 13-16 features run unrolled code in fp64 arithmetic (the
// fp32 G-form loses accuracy beyond 12), for either model dtype.
constexpr int kMaxUnrolledShapF64 = 16;

// Kernel variant by the model's longest path: every path has at most 8
// features, at most 12, at most 16 (SHAP values only), or any length up to a
// full bin (63).
constexpr int kQShort = 8;
constexpr int kQMid = 12;
constexpr int kQExt = 16;
constexpr int kQLong = 64;

// Private-tile launches (64-row tiles, one path per wave) of models with at
// most this many features keep rank tables of the row tile in LDS: per feature, the 64 row
// keys in ascending order and, for every rank, the mask of the rows below it.
// They serve the dead-pair test of a whole bin at once.
constexpr int kRankMaxM = 16;
inline size_t rank_table_bytes(int M) {
  return (size_t)M * 65 * (sizeof(uint64_t) + sizeof(int32_t));
}

// The launch shape of a model and row count: rows per tile, waves, private
// tiles, LDS strides and bytes, bin slices, and the kernel variant.
struct Plan {
  int RW = 0;
  int waves = 8;
  bool priv = false;
  int32_t sx = 0, sp = 0, width = 0;
  size_t lds = 0;
  int splits = 1;
  int min_splits = 1;    // slices enough for the occupancy target alone
  int split_step = 1;    // slice counts are multiples of this (XCD balance)
  int64_t tiles = 0;
  int qmax = kQLong;
  size_t rank_off = 0;   // LDS offset of the rank tables (0: none)
};

// Arguments of one gts_shap / gts_shap_interactions call.
struct KernelArgs {
  const gts_model* m;
  const void* blob;
  const float* X;
  int64_t rows;
  int64_t ld;
  void* phi;
  void* stream;   // hipStream_t
};

// One launcher per (dtype, kind); each lives in its own translation unit so
// the kernel variants compile in parallel.
gts_status launch_shap_f32(const KernelArgs& a, const Plan& p);
gts_status launch_shap_f64(const KernelArgs& a, const Plan& p);
gts_status launch_inter_f32(const KernelArgs& a, const Plan& p);
gts_status launch_inter_f64(const KernelArgs& a, const Plan& p);

}  // namespace gts
