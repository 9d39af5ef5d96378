// Internal declarations shared by the host (.cpp) and device (.hip) halves of
// libgts.  Not part of the public ABI.
#pragma once

#include <cstdint>

#include "gts.h"

namespace gts {

// Arrays of the device blob, indices into gts_model::off.  Elements are in
// bin order, the order gts_pack_paths produced: each bin is at most 64
// consecutive elements (one wave64 loads it with one element per lane), bins
// never mix output groups and are ordered by group.  A path is a root element
// followed by its feature elements; the root's zero-fraction slot holds the
// path's leaf value v (a root's own zero fraction is always 1 and unused).
// Within a bin, each path's zero-fraction elements come first (feature
// order), then its other elements rotated (see device_order in the host
// code); roots stay first.
enum BlobArray : int {
  kFeat = 0,       // int32[num_elements]   split feature; on a root -1 - (the
                   //                       path's zero-fraction elements)
  kLower = 1,      // float[num_elements]   range [lower, upper)
  kUpper = 2,      // float[num_elements]
  kZero = 3,       // T[num_elements]       zero fraction (leaf value on roots)
  kBinStart = 4,   // int32[num_bins+1]     element range of each bin
  kGroupBins = 5,  // int32[G+1]            bin range of each group
  kBias = 6,       // T[G]                  expected value per group
  kBlobArrays = 7
};

constexpr uint32_t kModelMagic = 0x31535447u;  // "GTS1"
constexpr int kMaxPathLen = 64;                // one wave64 holds a whole path
constexpr int64_t kBlobAlign = 256;

// Whether every launch of a model (SHAP and interaction values) runs one path
// per wave, i.e. picks 64-row tiles: the launch planner does so while a
// workgroup's X and phi tiles for 64 rows and the stages of its waves fit in
// 64 KB of LDS, and the interaction tile ((M+1)(M+2)/2 entries per row) is
// the larger, which holds up to M = 17 in fp32 and M = 11 in fp64.  For such
// models the order of a path's elements decides no same-step collisions.
inline bool one_path_per_wave(int32_t M, int32_t dtype) {
  return M <= (dtype == GTS_F64 ? 11 : 17);
}

// Thread-local error message; returns `status` for convenient tail calls.
gts_status fail(gts_status status, const char* fmt, ...)
    __attribute__((format(printf, 2, 3)));
void clear_error();

// Validates a descriptor produced by gts_model_layout.
gts_status check_model(const gts_model* m);

}  // namespace gts
