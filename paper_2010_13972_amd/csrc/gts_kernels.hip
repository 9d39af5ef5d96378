// Launch planning and the device entry points of libgts (gts_shap,
// gts_shap_interactions, gts_launch_config).  The kernels themselves are in
// gts_shap_kernel.h, instantiated by gts_shap_f32.hip, gts_shap_f64.hip,
// gts_inter_f32.hip and gts_inter_f64.hip.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <mutex>
#include <numeric>
#include <vector>

#include "gts_launch.h"
#include "gts_shap_kernel.h"

namespace gts {
namespace {

struct DeviceInfo {
  int cus = 256;
  int lds_per_block = 64 * 1024;
  int lds_per_cu = 160 * 1024;
};

DeviceInfo device_info() {
  static std::mutex mu;
  static std::vector<DeviceInfo> cache;
  static std::vector<char> have;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return DeviceInfo{};
  std::lock_guard<std::mutex> lock(mu);
  if ((int)cache.size() <= dev) {
    cache.resize(dev + 1);
    have.resize(dev + 1, 0);
  }
  if (!have[dev]) {
    DeviceInfo info;
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && n > 0)
      info.cus = n;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) == hipSuccess &&
        n > 0)
      info.lds_per_block = n;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor, dev) ==
            hipSuccess &&
        n > 0)
      info.lds_per_cu = n;
    info.lds_per_cu = std::max(info.lds_per_cu, info.lds_per_block);
    cache[dev] = info;
    have[dev] = 1;
  }
  return cache[dev];
}

inline int odd_at_least(int n) { return n | 1; }

template <typename T, bool INTER>
gts_status plan_launch(const gts_model* m, int64_t rows, const DeviceInfo& dev, Plan& plan) {
  const int M = m->num_features;
  const int G = m->num_groups;
  const int64_t width64 = INTER ? (int64_t)(M + 1) * (M + 1) : (int64_t)(M + 1);
  if (width64 > (1 << 30)) return fail(GTS_EINVAL, "M = %d is too large", M);
  const int32_t width = (int32_t)width64;
  const int32_t sx = odd_at_least(M);
  // interactions keep the upper triangle of each row's block in LDS
  const int32_t sp = odd_at_least(INTER ? (int32_t)((int64_t)(M + 1) * (M + 2) / 2) : width);
  // Row tile and accumulation.  If 64 rows with a private phi tile for each
  // of 4 waves fit in half a CU's LDS (two workgroups per CU), use them (no
  // contention, no atomics).  Otherwise 8 waves share one tile: the largest
  // RW whose tiles fit in 64 KB (several workgroups per CU), or, if that
  // would leave fewer than 8 rows per wave, 8 rows (then 4) using up to the
  // whole LDS of a workgroup.
  auto need = [&](int rw, int waves, bool priv) {
    const size_t tiles = (size_t)rw * ((size_t)sx * sizeof(float) +
                                       (priv ? (size_t)waves : 1) * (size_t)sp * sizeof(T));
    const size_t stage = rw == 64 ? sizeof(Stage<T, false>) : sizeof(Stage<T, true>);
    return ((tiles + 15) & ~(size_t)15) + (size_t)waves * stage;
  };
  int RW = 0;
  int waves = 8;
  bool priv = false;
  constexpr int64_t kSmallTile = 64 * 1024;  // leaves room for several workgroups per CU
  if ((int64_t)need(64, 4, true) <= std::min<int64_t>(kSmallTile, dev.lds_per_block)) {
    RW = 64;
    waves = 4;
    priv = true;
  } else {
    for (int cand : {64, 32, 16, 8}) {
      if ((int64_t)need(cand, 8, false) <= std::min<int64_t>(kSmallTile, dev.lds_per_block)) {
        RW = cand;
        break;
      }
    }
    if (INTER && RW == 0) {
      // Interaction values: 16 waves (the kernel's registers allow one
      // workgroup of them per CU) on the largest tile of 16, 8 or 4 rows the
      // LDS of a workgroup holds.
      for (int cand : {16, 8, 4}) {
        if ((int64_t)need(cand, 16, false) <= dev.lds_per_block) {
          RW = cand;
          waves = 16;
          break;
        }
      }
    }
    if (RW == 0 && (int64_t)need(8, 8, false) <= dev.lds_per_block) RW = 8;
    if (RW == 0 && (int64_t)need(4, 8, false) <= dev.lds_per_block) RW = 4;
    // Waves per workgroup for a shared tile of RW <= 16 rows: as many waves
    // per CU as the LDS allows, up to 24 (the VGPR budget of the SHAP
    // kernels).
    if (!INTER && RW != 0 && RW <= 16) {
      const int cap = 24;
      int best = 0;
      for (int w : {8, 12, 16}) {
        const int64_t n = need(RW, w, false);
        if (n > dev.lds_per_block) continue;
        const int per_cu = (int)std::min<int64_t>(cap, w * (dev.lds_per_cu / n));
        if (per_cu > best) {
          best = per_cu;
          waves = w;
        }
      }
    }
  }
  if (RW == 0) return fail(GTS_EINVAL, "M = %d needs more LDS than a workgroup has", M);
  size_t lds = need(RW, waves, priv);
  // rank tables for the bin-wide dead-pair test of one-path-per-wave launches
  size_t rank_off = 0;
  if (RW == 64 && priv && M <= kRankMaxM) {
    rank_off = (lds + 7) & ~(size_t)7;
    lds = rank_off + rank_table_bytes(M);
  }
  // Bin slices per (row tile, group) when there are too few tiles to fill
  // the GPU.  Every slice adds its tile to phi atomically, so a slice costs
  // rows x width atomic adds.  SHAP values (short phi rows): enough
  // workgroups for two rounds of every CU at the occupancy the LDS allows,
  // or more, up to 128 slices, while every wave still gets 8 bins or more
  // (finer slices even out the last rounds); (group, slice) units a multiple
  // of the 8 XCDs.  Interaction values ((M+1)^2 per row): at most one round,
  // since there the adds outweigh the balance.
  const int64_t tiles = (rows + RW - 1) / RW;
  const int64_t base = tiles * G;
  const int64_t per_cu = std::max<int64_t>(1, std::min<int64_t>(8, dev.lds_per_cu / (int64_t)lds));
  const int64_t bins_per_group = std::max<int64_t>(1, m->num_bins / G);
  int splits = 1;
  int min_splits = 1;
  int split_step = 1;
  if constexpr (INTER) {
    const int64_t round = per_cu * dev.cus;
    if (2 * base <= round)
      splits = (int)std::max<int64_t>(1, std::min<int64_t>(round / base, bins_per_group));
    min_splits = splits;
  } else {
    const int64_t target = 2 * per_cu * dev.cus;
    if (base < target) {
      int64_t want = (target + base - 1) / base;
      const int64_t step = 8 / std::gcd(G, 8);
      want = (want + step - 1) / step * step;
      const int64_t fine = std::min<int64_t>(128, bins_per_group / (8 * waves)) / step * step;
      min_splits = (int)std::max<int64_t>(1, std::min<int64_t>(want, bins_per_group));
      want = std::max(want, fine);
      splits = (int)std::max<int64_t>(1, std::min<int64_t>(want, bins_per_group));
      split_step = (int)step;
    }
    min_splits = std::min(min_splits, splits);
  }
  plan.RW = RW;
  plan.waves = waves;
  plan.priv = priv;
  plan.sx = sx;
  plan.sp = sp;
  plan.width = width;
  plan.lds = lds;
  plan.rank_off = rank_off;
  plan.splits = splits;
  plan.min_splits = min_splits;
  plan.split_step = split_step;
  plan.tiles = tiles;
  // the kernel variant: the model's longest path, in features
  const int qmax = std::max(0, m->max_path_len - 1);
  plan.qmax = qmax <= kQShort ? kQShort
              : (!INTER && qmax <= kMaxUnrolledShap) ? kQMid
              : (!INTER && qmax <= kMaxUnrolledShapF64) ? kQExt
                                                        : kQLong;
  return GTS_OK;
}

gts_status launch(const gts_model* m, const void* blob, const float* X, int64_t rows,
                  int64_t ld, void* phi, void* stream, bool inter) {
  Plan plan;
  const DeviceInfo dev = device_info();
  gts_status st;
  if (m->dtype == GTS_F64)
    st = inter ? plan_launch<double, true>(m, rows, dev, plan)
               : plan_launch<double, false>(m, rows, dev, plan);
  else
    st = inter ? plan_launch<float, true>(m, rows, dev, plan)
               : plan_launch<float, false>(m, rows, dev, plan);
  if (st != GTS_OK) return st;
  const KernelArgs a{m, blob, X, rows, ld, phi, stream};
  if (m->dtype == GTS_F64) return inter ? launch_inter_f64(a, plan) : launch_shap_f64(a, plan);
  return inter ? launch_inter_f32(a, plan) : launch_shap_f32(a, plan);
}

gts_status entry(const gts_model* model, const void* d_model, const float* d_X, int64_t rows,
                 int64_t ld_x, void* d_phi, void* stream, bool inter) {
  clear_error();
  gts_status st = check_model(model);
  if (st != GTS_OK) return st;
  if (rows < 0) return fail(GTS_EINVAL, "rows must be >= 0");
  if (rows == 0) return GTS_OK;
  if (d_model == nullptr || d_X == nullptr || d_phi == nullptr)
    return fail(GTS_EINVAL, "device pointers must not be NULL");
  if (ld_x < model->num_features) return fail(GTS_EINVAL, "ld_x < num_features");
  return launch(model, d_model, d_X, rows, ld_x, d_phi, stream, inter);
}

}  // namespace
}  // namespace gts

extern "C" gts_status gts_launch_config(const gts_model* model, int64_t rows,
                                        int32_t interactions, gts_launch* out) {
  using namespace gts;
  clear_error();
  if (out == nullptr) return fail(GTS_EINVAL, "out must not be NULL");
  gts_status st = check_model(model);
  if (st != GTS_OK) return st;
  if (rows < 0) return fail(GTS_EINVAL, "rows must be >= 0");
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return fail(GTS_EDEVICE, "no HIP device");
  Plan plan;
  const DeviceInfo info = device_info();
  const int64_t r = rows > 0 ? rows : 1;
  if (model->dtype == GTS_F64)
    st = interactions ? plan_launch<double, true>(model, r, info, plan)
                      : plan_launch<double, false>(model, r, info, plan);
  else
    st = interactions ? plan_launch<float, true>(model, r, info, plan)
                      : plan_launch<float, false>(model, r, info, plan);
  if (st != GTS_OK) return st;
  out->rows_per_tile = plan.RW;
  out->waves = plan.waves;
  out->private_tiles = plan.priv ? 1 : 0;
  out->slices = plan.splits;
  out->workgroups = rows > 0 ? plan.tiles * model->num_groups * plan.splits : 0;
  out->lds_bytes = (int64_t)plan.lds;
  return GTS_OK;
}

extern "C" gts_status gts_shap(const gts_model* model, const void* d_model, const float* d_X,
                               int64_t rows, int64_t ld_x, void* d_phi, void* stream) {
  return gts::entry(model, d_model, d_X, rows, ld_x, d_phi, stream, false);
}

extern "C" gts_status gts_shap_interactions(const gts_model* model, const void* d_model,
                                            const float* d_X, int64_t rows, int64_t ld_x,
                                            void* d_phi, void* stream) {
  return gts::entry(model, d_model, d_X, rows, ld_x, d_phi, stream, true);
}
