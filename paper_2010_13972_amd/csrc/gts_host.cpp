// Host half of libgts: argument checking, path extraction with duplicate
// merging (Sections 3.1-3.2), bin packing (Section 3.3) and the device
// layout.  Compiled without floating-point contraction so that the extracted
// zero fractions and the bias are reproducible bit for bit.
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <functional>
#include <limits>
#include <new>
#include <vector>

#include "gts_internal.h"

namespace gts {

static thread_local char g_error[512];

gts_status fail(gts_status status, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(g_error, sizeof(g_error), fmt, ap);
  va_end(ap);
  return status;
}

void clear_error() { g_error[0] = '\0'; }

gts_status check_model(const gts_model* m) {
  if (m == nullptr) return fail(GTS_EINVAL, "model descriptor is NULL");
  if (m->magic != kModelMagic)
    return fail(GTS_EINVAL, "model descriptor was not produced by gts_model_layout");
  if (m->dtype != GTS_F32 && m->dtype != GTS_F64)
    return fail(GTS_EINVAL, "model dtype %d is not GTS_F32 or GTS_F64", m->dtype);
  if (m->num_features < 1 || m->num_groups < 1)
    return fail(GTS_EINVAL, "model has M=%d, G=%d", m->num_features, m->num_groups);
  if (m->max_path_len < 0 || m->max_path_len > kMaxPathLen)
    return fail(GTS_EINVAL, "model max path length %d out of range", m->max_path_len);
  return GTS_OK;
}

namespace {

// One split on the way from the root to a leaf.
struct Split {
  int32_t feature;
  float lower, upper;
  double zero_fraction;
};

inline double cover_ratio(double child, double parent) {
  return parent > 0.0 ? child / parent : 0.0;
}

gts_status validate_ensemble(const gts_ensemble* e) {
  if (e == nullptr) return fail(GTS_EINVAL, "ensemble is NULL");
  if (e->num_features < 1) return fail(GTS_EINVAL, "num_features must be >= 1");
  if (e->num_groups < 1) return fail(GTS_EINVAL, "num_groups must be >= 1");
  if (e->num_trees < 0) return fail(GTS_EINVAL, "num_trees must be >= 0");
  if (e->num_trees == 0) return GTS_OK;
  if (!e->tree_node_offsets || !e->tree_group || !e->left || !e->right ||
      !e->feature || !e->threshold || !e->cover || !e->value)
    return fail(GTS_EINVAL, "an ensemble array pointer is NULL");
  if (e->tree_node_offsets[0] != 0)
    return fail(GTS_EINVAL, "tree_node_offsets[0] must be 0");
  for (int64_t t = 0; t < e->num_trees; ++t) {
    const int64_t a = e->tree_node_offsets[t], b = e->tree_node_offsets[t + 1];
    if (b <= a) return fail(GTS_EINVAL, "tree %lld has no nodes", (long long)t);
    if (b - a > std::numeric_limits<int32_t>::max())
      return fail(GTS_EINVAL, "tree %lld has too many nodes", (long long)t);
    const int32_t g = e->tree_group[t];
    if (g < 0 || g >= e->num_groups)
      return fail(GTS_EINVAL, "tree %lld has group %d outside [0, %d)", (long long)t, g,
                  e->num_groups);
  }
  if (e->tree_node_offsets[e->num_trees] != e->num_nodes)
    return fail(GTS_EINVAL, "tree_node_offsets[T] != num_nodes");
  return GTS_OK;
}

// Depth-first walk of one tree (left child first).  Calls leaf(node, splits,
// count) at every leaf.  Rejects bad children, revisits and bad node data.
template <typename LeafFn>
gts_status walk_tree(const gts_ensemble* e, int64_t t, std::vector<Split>& path,
                     std::vector<unsigned char>& seen, LeafFn&& leaf) {
  const int64_t base = e->tree_node_offsets[t];
  const int32_t n = (int32_t)(e->tree_node_offsets[t + 1] - base);
  seen.assign((size_t)n, 0);
  struct Frame { int32_t node; int32_t depth; Split into; };
  std::vector<Frame> stack;
  stack.push_back(Frame{0, 0, Split{}});
  while (!stack.empty()) {
    const Frame fr = stack.back();
    stack.pop_back();
    const int32_t node = fr.node;
    if (seen[(size_t)node])
      return fail(GTS_EINVAL, "tree %lld: node %d reached twice (cycle or shared child)",
                  (long long)t, node);
    seen[(size_t)node] = 1;
    path.resize((size_t)fr.depth);
    if (fr.depth > 0) path[(size_t)fr.depth - 1] = fr.into;
    const int64_t gi = base + node;
    const double r = e->cover[gi];
    if (!(r >= 0.0) || !std::isfinite(r))
      return fail(GTS_EINVAL, "tree %lld node %d: cover must be finite and >= 0",
                  (long long)t, node);
    const int32_t a = e->left[gi], b = e->right[gi];
    if (a < 0 && b < 0) {
      if (!std::isfinite(e->value[gi]))
        return fail(GTS_EINVAL, "tree %lld leaf %d: value is not finite", (long long)t, node);
      gts_status st = leaf(node, path);
      if (st != GTS_OK) return st;
      continue;
    }
    if (a < 0 || b < 0 || a >= n || b >= n)
      return fail(GTS_EINVAL, "tree %lld node %d: child index out of range", (long long)t,
                  node);
    const int32_t d = e->feature[gi];
    if (d < 0 || d >= e->num_features)
      return fail(GTS_EINVAL, "tree %lld node %d: feature %d outside [0, %d)", (long long)t,
                  node, d, e->num_features);
    const float th = e->threshold[gi];
    if (std::isnan(th))
      return fail(GTS_EINVAL, "tree %lld node %d: threshold is NaN", (long long)t, node);
    const double ra = e->cover[base + a], rb = e->cover[base + b];
    const float inf = std::numeric_limits<float>::infinity();
    // right child pushed first so the left child (x < t) is visited first
    stack.push_back(Frame{b, fr.depth + 1, Split{d, th, inf, cover_ratio(rb, r)}});
    stack.push_back(Frame{a, fr.depth + 1, Split{d, -inf, th, cover_ratio(ra, r)}});
  }
  return GTS_OK;
}

}  // namespace
}  // namespace gts

using namespace gts;

extern "C" {

const char* gts_last_error(void) { return g_error; }

const char* gts_version(void) { return "gts 0.1 (gfx950)"; }

gts_status gts_extract_paths(const gts_ensemble* ens, gts_path_element* out,
                             int64_t capacity, int64_t* num_elements,
                             int64_t* num_paths, double* bias) {
  clear_error();
  if (num_elements == nullptr || num_paths == nullptr)
    return fail(GTS_EINVAL, "num_elements and num_paths must not be NULL");
  if (capacity < 0) return fail(GTS_EINVAL, "capacity must be >= 0");
  if (out == nullptr && capacity > 0) return fail(GTS_EINVAL, "out is NULL but capacity > 0");
  gts_status st = validate_ensemble(ens);
  if (st != GTS_OK) return st;
  try {
    if (bias)
      for (int32_t g = 0; g < ens->num_groups; ++g) bias[g] = 0.0;
    int64_t n = 0, paths = 0;
    std::vector<Split> path, sorted;
    std::vector<unsigned char> seen;
    for (int64_t t = 0; t < ens->num_trees; ++t) {
      const int64_t base = ens->tree_node_offsets[t];
      const int32_t group = ens->tree_group[t];
      st = walk_tree(ens, t, path, seen, [&](int32_t leaf, const std::vector<Split>& sp) {
        const double v = ens->value[base + leaf];
        // Section 3.2: order by feature (stable: repeats stay root-to-leaf),
        // then combine consecutive repeats into one element.
        sorted.assign(sp.begin(), sp.end());
        std::stable_sort(sorted.begin(), sorted.end(),
                         [](const Split& x, const Split& y) { return x.feature < y.feature; });
        size_t m = 0;
        for (size_t i = 0; i < sorted.size(); ++i) {
          if (m > 0 && sorted[m - 1].feature == sorted[i].feature) {
            Split& acc = sorted[m - 1];
            if (sorted[i].lower > acc.lower) acc.lower = sorted[i].lower;
            if (sorted[i].upper < acc.upper) acc.upper = sorted[i].upper;
            acc.zero_fraction = acc.zero_fraction * sorted[i].zero_fraction;
          } else {
            sorted[m] = sorted[i];
            sorted[m].zero_fraction = 1.0 * sorted[i].zero_fraction;
            ++m;
          }
        }
        sorted.resize(m);
        if (bias) {
          double prod = 1.0;
          for (size_t i = 0; i < m; ++i) prod = prod * sorted[i].zero_fraction;
          bias[group] += v * prod;
        }
        const float inf = std::numeric_limits<float>::infinity();
        for (size_t i = 0; i <= m; ++i) {
          if (n < capacity) {
            gts_path_element& el = out[n];
            el.path_idx = paths;
            el.group = group;
            el.v = v;
            if (i == 0) {
              el.feature_idx = -1;
              el.lower = -inf;
              el.upper = inf;
              el.zero_fraction = 1.0;
            } else {
              el.feature_idx = sorted[i - 1].feature;
              el.lower = sorted[i - 1].lower;
              el.upper = sorted[i - 1].upper;
              el.zero_fraction = sorted[i - 1].zero_fraction;
            }
          }
          ++n;
        }
        ++paths;
        return GTS_OK;
      });
      if (st != GTS_OK) return st;
    }
    *num_elements = n;
    *num_paths = paths;
    if (n > capacity && out != nullptr)
      return fail(GTS_EBUFSIZE, "capacity %lld < %lld elements", (long long)capacity,
                  (long long)n);
    return GTS_OK;
  } catch (const std::bad_alloc&) {
    return fail(GTS_ENOMEM, "host allocation failed");
  }
}

}  // extern "C"

namespace gts {
namespace {

struct PathRef {
  int64_t first;  // element index of the root
  int32_t size;   // path length, root included
  int32_t group;
};

gts_status parse_paths(const gts_path_element* el, int64_t n, std::vector<PathRef>& paths,
                       int32_t max_len, int32_t num_groups /* 0 = unchecked */,
                       int32_t num_features /* 0 = unchecked */) {
  paths.clear();
  if (n == 0) return GTS_OK;
  if (el == nullptr) return fail(GTS_EINVAL, "elements pointer is NULL");
  if (el[0].feature_idx != -1)
    return fail(GTS_EINVAL, "element 0 is not a root element (feature_idx -1)");
  for (int64_t i = 0; i < n; ++i) {
    const gts_path_element& e = el[i];
    if (e.feature_idx == -1) {
      if (!paths.empty() && paths.back().size > max_len)
        return fail(GTS_EPATHLEN, "path at element %lld has length %d > %d",
                    (long long)paths.back().first, paths.back().size, max_len);
      paths.push_back(PathRef{i, 1, e.group});
      if (num_groups > 0 && (e.group < 0 || e.group >= num_groups))
        return fail(GTS_EINVAL, "element %lld: group %d outside [0, %d)", (long long)i,
                    e.group, num_groups);
      continue;
    }
    PathRef& p = paths.back();
    const gts_path_element& root = el[p.first];
    if (e.feature_idx < -1 || (num_features > 0 && e.feature_idx >= num_features))
      return fail(GTS_EINVAL, "element %lld: feature %d out of range", (long long)i,
                  e.feature_idx);
    if (e.path_idx != root.path_idx || e.group != root.group)
      return fail(GTS_EINVAL, "element %lld does not belong to the path started at %lld",
                  (long long)i, (long long)p.first);
    ++p.size;
  }
  if (paths.back().size > max_len)
    return fail(GTS_EPATHLEN, "path at element %lld has length %d > %d",
                (long long)paths.back().first, paths.back().size, max_len);
  return GTS_OK;
}

// Min-heap of bin numbers.
using BinHeap = std::vector<int64_t>;
inline void heap_push(BinHeap& h, int64_t b) {
  h.push_back(b);
  std::push_heap(h.begin(), h.end(), std::greater<int64_t>());
}
inline int64_t heap_pop(BinHeap& h) {
  std::pop_heap(h.begin(), h.end(), std::greater<int64_t>());
  const int64_t b = h.back();
  h.pop_back();
  return b;
}

// Leftmost open bin with residual >= s, over a max-segment-tree of residuals.
struct FirstFitTree {
  int64_t size = 1;
  std::vector<int32_t> t;
  explicit FirstFitTree(int64_t n) {
    while (size < n) size <<= 1;
    t.assign((size_t)(2 * size), 0);
  }
  void set(int64_t i, int32_t v) {
    int64_t k = i + size;
    t[(size_t)k] = v;
    for (k >>= 1; k >= 1; k >>= 1) t[(size_t)k] = std::max(t[(size_t)(2 * k)], t[(size_t)(2 * k + 1)]);
  }
  int64_t leftmost_at_least(int32_t s) const {
    if (t[1] < s) return -1;
    int64_t k = 1;
    while (k < size) k = (t[(size_t)(2 * k)] >= s) ? 2 * k : 2 * k + 1;
    return k - size;
  }
};

}  // namespace
}  // namespace gts

extern "C" gts_status gts_pack_paths(const gts_path_element* elems, int64_t num_elements,
                                     int32_t bin_capacity, int32_t alg,
                                     gts_path_element* packed, int64_t* bin_offsets,
                                     int64_t offsets_capacity, int64_t* num_bins) {
  clear_error();
  if (num_bins == nullptr) return fail(GTS_EINVAL, "num_bins must not be NULL");
  if (num_elements < 0) return fail(GTS_EINVAL, "num_elements must be >= 0");
  if (bin_capacity < 1 || bin_capacity > kMaxPathLen)
    return fail(GTS_EINVAL, "bin_capacity %d outside [1, %d]", bin_capacity, kMaxPathLen);
  if (alg < GTS_PACK_BFD || alg > GTS_PACK_NONE)
    return fail(GTS_EINVAL, "unknown packing algorithm %d", alg);
  if (offsets_capacity < 0 || (offsets_capacity > 0 && bin_offsets == nullptr))
    return fail(GTS_EINVAL, "bad bin_offsets / offsets_capacity");
  if (offsets_capacity > 0 && packed == nullptr && num_elements > 0)
    return fail(GTS_EINVAL, "packed must not be NULL when offsets are requested");
  try {
    std::vector<PathRef> paths;
    gts_status st = parse_paths(elems, num_elements, paths, bin_capacity, 0, 0);
    if (st != GTS_OK) return st;
    const int64_t P = (int64_t)paths.size();
    // processing order: by group, then per algorithm
    std::vector<int64_t> order((size_t)P);
    for (int64_t i = 0; i < P; ++i) order[(size_t)i] = i;
    const bool decreasing = (alg == GTS_PACK_BFD || alg == GTS_PACK_FFD);
    std::stable_sort(order.begin(), order.end(), [&](int64_t a, int64_t b) {
      const PathRef &x = paths[(size_t)a], &y = paths[(size_t)b];
      if (x.group != y.group) return x.group < y.group;
      if (decreasing && x.size != y.size) return x.size > y.size;
      return a < b;
    });
    std::vector<int64_t> bin_of((size_t)P);
    std::vector<int32_t> resid;
    int64_t K = 0;
    size_t i = 0;
    while (i < order.size()) {
      const int32_t g = paths[(size_t)order[i]].group;
      size_t j = i;
      while (j < order.size() && paths[(size_t)order[j]].group == g) ++j;
      const int64_t first_bin = K;
      if (alg == GTS_PACK_BFD) {
        std::vector<BinHeap> by_resid((size_t)bin_capacity + 1);
        for (size_t k = i; k < j; ++k) {
          const int32_t s = paths[(size_t)order[k]].size;
          int64_t b = -1;
          int32_t r = s;
          for (; r <= bin_capacity; ++r)
            if (!by_resid[(size_t)r].empty()) { b = heap_pop(by_resid[(size_t)r]); break; }
          if (b < 0) {
            b = K++;
            r = bin_capacity;
          }
          const int32_t left = r - s;
          if (left > 0) heap_push(by_resid[(size_t)left], b);
          bin_of[(size_t)order[k]] = b;
        }
      } else if (alg == GTS_PACK_FFD) {
        FirstFitTree tree((int64_t)(j - i));
        int64_t opened = 0;
        for (size_t k = i; k < j; ++k) {
          const int32_t s = paths[(size_t)order[k]].size;
          int64_t local = tree.leftmost_at_least(s);
          if (local < 0) {
            local = opened++;
            resid.resize((size_t)(first_bin + opened));
            resid[(size_t)(first_bin + local)] = bin_capacity;
          }
          const int64_t b = first_bin + local;
          resid[(size_t)b] -= s;
          tree.set(local, resid[(size_t)b]);
          bin_of[(size_t)order[k]] = b;
        }
        K = first_bin + opened;
      } else if (alg == GTS_PACK_NF) {
        int32_t r = 0;
        for (size_t k = i; k < j; ++k) {
          const int32_t s = paths[(size_t)order[k]].size;
          if (K == first_bin || r < s) {
            ++K;
            r = bin_capacity;
          }
          r -= s;
          bin_of[(size_t)order[k]] = K - 1;
        }
      } else {
        for (size_t k = i; k < j; ++k) bin_of[(size_t)order[k]] = K++;
      }
      i = j;
    }
    *num_bins = K;
    if (offsets_capacity == 0) return GTS_OK;
    if (offsets_capacity < K + 1)
      return fail(GTS_EBUFSIZE, "offsets_capacity %lld < num_bins + 1 = %lld",
                  (long long)offsets_capacity, (long long)(K + 1));
    // lay bins out in order; inside a bin, paths in placement order
    std::vector<int64_t> count((size_t)K + 1, 0);
    for (int64_t p = 0; p < P; ++p) count[(size_t)bin_of[(size_t)p] + 1] += paths[(size_t)p].size;
    for (int64_t b = 0; b < K; ++b) count[(size_t)b + 1] += count[(size_t)b];
    for (int64_t b = 0; b <= K; ++b) bin_offsets[b] = count[(size_t)b];
    std::vector<int64_t> cursor(count.begin(), count.end() - 1);
    for (size_t k = 0; k < order.size(); ++k) {
      const PathRef& p = paths[(size_t)order[k]];
      const int64_t b = bin_of[(size_t)order[k]];
      std::memcpy(packed + cursor[(size_t)b], elems + p.first, sizeof(gts_path_element) * (size_t)p.size);
      cursor[(size_t)b] += p.size;
    }
    return GTS_OK;
  } catch (const std::bad_alloc&) {
    return fail(GTS_ENOMEM, "host allocation failed");
  }
}

extern "C" gts_status gts_model_layout(const gts_path_element* packed, int64_t num_elements,
                                       const int64_t* bin_offsets, int64_t num_bins,
                                       int32_t num_features, int32_t num_groups,
                                       const double* bias, int32_t dtype, gts_model* model,
                                       void* host_blob, int64_t blob_capacity) {
  clear_error();
  if (model == nullptr) return fail(GTS_EINVAL, "model must not be NULL");
  if (num_features < 1 || num_groups < 1)
    return fail(GTS_EINVAL, "num_features and num_groups must be >= 1");
  if (dtype != GTS_F32 && dtype != GTS_F64) return fail(GTS_EINVAL, "unknown dtype %d", dtype);
  if (num_elements < 0 || num_bins < 0) return fail(GTS_EINVAL, "negative size");
  if (num_elements >= std::numeric_limits<int32_t>::max())
    return fail(GTS_EINVAL, "too many path elements for 32-bit device indices");
  if (bin_offsets == nullptr) return fail(GTS_EINVAL, "bin_offsets must not be NULL");
  if (bias == nullptr) return fail(GTS_EINVAL, "bias must not be NULL");
  if (blob_capacity < 0 || (blob_capacity > 0 && host_blob == nullptr))
    return fail(GTS_EINVAL, "bad host_blob / blob_capacity");
  try {
    std::vector<PathRef> paths;
    gts_status st = parse_paths(packed, num_elements, paths, kMaxPathLen, num_groups, num_features);
    if (st != GTS_OK) return st;
    if (bin_offsets[0] != 0 || bin_offsets[num_bins] != num_elements)
      return fail(GTS_EINVAL, "bin_offsets must run from 0 to num_elements");
    // every bin starts on a root element and holds paths of one group
    std::vector<int32_t> bin_group((size_t)num_bins);
    {
      size_t p = 0;
      for (int64_t b = 0; b < num_bins; ++b) {
        const int64_t a = bin_offsets[b], e = bin_offsets[b + 1];
        if (e < a || e - a > kMaxPathLen)
          return fail(GTS_EINVAL, "bin %lld spans %lld elements", (long long)b, (long long)(e - a));
        if (a == e) return fail(GTS_EINVAL, "bin %lld is empty", (long long)b);
        while (p < paths.size() && paths[p].first < a) ++p;
        if (p >= paths.size() || paths[p].first != a)
          return fail(GTS_EINVAL, "bin %lld does not start on a path root", (long long)b);
        bin_group[(size_t)b] = paths[p].group;
        for (size_t q = p; q < paths.size() && paths[q].first < e; ++q) {
          if (paths[q].first + paths[q].size > e)
            return fail(GTS_EINVAL, "a path crosses the end of bin %lld", (long long)b);
          if (paths[q].group != bin_group[(size_t)b])
            return fail(GTS_EINVAL, "bin %lld mixes output groups", (long long)b);
        }
        if (b > 0 && bin_group[(size_t)b] < bin_group[(size_t)b - 1])
          return fail(GTS_EINVAL, "bins must be ordered by group");
      }
    }
    const int64_t P = (int64_t)paths.size();
    const int64_t G = num_groups;
    const size_t ts = dtype == GTS_F64 ? sizeof(double) : sizeof(float);
    int64_t sizes[kBlobArrays];
    sizes[kFeat] = 4 * num_elements;
    sizes[kLower] = 4 * num_elements;
    sizes[kUpper] = 4 * num_elements;
    sizes[kZero] = (int64_t)ts * num_elements;
    sizes[kBinStart] = 4 * (num_bins + 1);
    sizes[kGroupBins] = 4 * (G + 1);
    sizes[kBias] = (int64_t)ts * G;
    gts_model m;
    std::memset(&m, 0, sizeof(m));
    m.magic = kModelMagic;
    m.dtype = dtype;
    m.num_features = num_features;
    m.num_groups = num_groups;
    m.num_elements = num_elements;
    m.num_paths = P;
    m.num_bins = num_bins;
    int64_t cur = 0;
    for (int k = 0; k < kBlobArrays; ++k) {
      m.off[k] = cur;
      cur += (sizes[k] + kBlobAlign - 1) / kBlobAlign * kBlobAlign;
    }
    m.bytes = cur > 0 ? cur : kBlobAlign;
    int32_t maxlen = 0;
    for (const PathRef& p : paths) maxlen = std::max(maxlen, p.size);
    m.max_path_len = maxlen;
    *model = m;
    if (host_blob == nullptr) return GTS_OK;
    if (blob_capacity < m.bytes)
      return fail(GTS_EBUFSIZE, "blob_capacity %lld < %lld bytes", (long long)blob_capacity,
                  (long long)m.bytes);
    char* blob = static_cast<char*>(host_blob);
    std::memset(blob, 0, (size_t)m.bytes);
    int32_t* feat = reinterpret_cast<int32_t*>(blob + m.off[kFeat]);
    float* lower = reinterpret_cast<float*>(blob + m.off[kLower]);
    float* upper = reinterpret_cast<float*>(blob + m.off[kUpper]);
    for (int64_t i = 0; i < num_elements; ++i) {
      feat[i] = packed[i].feature_idx;
      lower[i] = packed[i].lower;
      upper[i] = packed[i].upper;
    }
    int32_t* bstart = reinterpret_cast<int32_t*>(blob + m.off[kBinStart]);
    int32_t* gbins = reinterpret_cast<int32_t*>(blob + m.off[kGroupBins]);
    for (int64_t b = 0; b <= num_bins; ++b) bstart[b] = (int32_t)bin_offsets[b];
    for (int64_t g = 0; g <= G; ++g) gbins[g] = 0;
    for (int64_t b = 0; b < num_bins; ++b) gbins[bin_group[(size_t)b] + 1] += 1;
    for (int64_t g = 0; g < G; ++g) gbins[g + 1] += gbins[g];
    if (dtype == GTS_F64) {
      double* z = reinterpret_cast<double*>(blob + m.off[kZero]);
      double* bb = reinterpret_cast<double*>(blob + m.off[kBias]);
      for (int64_t i = 0; i < num_elements; ++i)
        z[i] = packed[i].feature_idx == -1 ? packed[i].v : packed[i].zero_fraction;
      for (int64_t g = 0; g < G; ++g) bb[g] = bias[g];
    } else {
      float* z = reinterpret_cast<float*>(blob + m.off[kZero]);
      float* bb = reinterpret_cast<float*>(blob + m.off[kBias]);
      for (int64_t i = 0; i < num_elements; ++i)
        z[i] = (float)(packed[i].feature_idx == -1 ? packed[i].v : packed[i].zero_fraction);
      for (int64_t g = 0; g < G; ++g) bb[g] = (float)bias[g];
    }
    return GTS_OK;
  } catch (const std::bad_alloc&) {
    return fail(GTS_ENOMEM, "host allocation failed");
  }
}
