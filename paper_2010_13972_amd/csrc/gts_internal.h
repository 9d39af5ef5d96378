// Internal declarations shared by the host (.cpp) and device (.hip) halves of
// libgts.  Not part of the public ABI.
#pragma once

#include <cstdint>

#include "gts.h"

namespace gts {

// Arrays of the device blob, indices into gts_model::off.  Elements are in
// bin order (the order gts_pack_paths produced); per-path arrays are in
// "row-lane order": grouped by output group, then by non-increasing path
// length, so consecutive paths have equal or similar lengths.
enum BlobArray : int {
  kFeat = 0,       // int32[num_elements]   split feature, -1 on root elements
  kLower = 1,      // float[num_elements]   range [lower, upper)
  kUpper = 2,      // float[num_elements]
  kZero = 3,       // T[num_elements]       zero fraction
  kPathFirst = 4,  // int32[num_paths]      element index of the path's root
  kPathLen = 5,    // int32[num_paths]      path length, root included
  kPathV = 6,      // T[num_paths]          leaf value
  kGroupPaths = 7, // int32[G+1]            path range of each group
  kBinStart = 8,   // int32[num_bins+1]     element range of each bin
  kGroupBins = 9,  // int32[G+1]            bin range of each group
  kBias = 10,      // T[G]                  expected value per group
  kBlobArrays = 11
};

constexpr uint32_t kModelMagic = 0x31535447u;  // "GTS1"
constexpr int kMaxPathLen = 64;                // one wave64 holds a whole path
constexpr int64_t kBlobAlign = 256;

// Thread-local error message; returns `status` for convenient tail calls.
gts_status fail(gts_status status, const char* fmt, ...)
    __attribute__((format(printf, 2, 3)));
void clear_error();

// Validates a descriptor produced by gts_model_layout.
gts_status check_model(const gts_model* m);

}  // namespace gts
