// Path extraction on the GPU (Sections 3.1-3.2): the unique root-to-leaf
// paths of an ensemble whose node arrays are in device memory, with repeated
// features merged, written in the canonical order of gts_extract_paths and
// bit for bit equal to it, plus the bias of every output group.
//
// One thread per node validates it and links it to its parent; one thread
// per leaf then walks up to its tree's root, which
//   - counts the leaves under every node (atomic increments on the way up),
//   - gives the leaf's rank in depth-first preorder with the left child
//     first: the number of leaves under every left sibling it passes,
//   - collects the splits of its path, which it replays from the root down to
//     merge repeated features (ranges intersected, zero fractions multiplied
//     in root-to-leaf order, features kept in ascending order).
// Scans over trees and paths place every path; each tree sums its paths' bias
// terms v * prod(z) in path order and each group its trees' sums in tree
// order, the order the host uses.
//
// Compiled without floating-point contraction: the cover ratios (IEEE
// division), their products and the bias sums round exactly as on the host.
#include <hip/hip_runtime.h>

#include <rocprim/device/device_scan.hpp>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <mutex>
#include <vector>

#include "gts_internal.h"

namespace gts {
namespace {

constexpr int kMaxDepth = 256;      // longest root-to-leaf chain of splits
constexpr int kMaxMerged = kMaxPathLen - 1;  // features a merged path may hold
constexpr int kThreads = 256;

// Error codes recorded by the kernels (first one wins).
enum ExtractError : int {
  kOk = 0,
  kBadOffsets = 1,
  kBadGroup = 2,
  kBadCover = 3,
  kBadValue = 4,
  kBadChild = 5,
  kBadFeature = 6,
  kNanThreshold = 7,
  kTwoParents = 8,
  kRootHasParent = 9,
  kTooDeep = 10,
  kTooLong = 11
};

struct DevEnsemble {
  const int64_t* __restrict__ off;
  const int32_t* __restrict__ group;
  const int32_t* __restrict__ left;
  const int32_t* __restrict__ right;
  const int32_t* __restrict__ feature;
  const float* __restrict__ threshold;
  const double* __restrict__ cover;
  const double* __restrict__ value;
  int64_t T;
  int64_t N;
  int32_t M;
  int32_t G;
};

// Workspace arrays (every array 256-byte aligned in the caller's buffer).
struct Work {
  int32_t* err;        // [4] code, tree, node, unused
  int32_t* parent;     // [N] local index of the parent, -1 for none
  int32_t* npar;       // [N] number of parents
  int32_t* leaves;     // [N] reachable leaves under the node
  int32_t* rank;       // [N] on a reachable leaf: preorder rank in its tree, else -1
  int32_t* merged;     // [N] on a reachable leaf: merged path length (features)
  int64_t* tree_leaves;  // [T+1] reachable leaves per tree
  int64_t* tree_off;     // [T+1] their exclusive scan: first path of every tree
  int64_t* path_leaf;    // [N] leaf node (global index) of each path
  int64_t* path_elems;   // [N+1] elements per path
  int64_t* elem_off;     // [N+1] their exclusive scan: first element of every path
  double* term;          // [N] bias term of each path
  double* tree_sum;      // [T] bias terms summed per tree
  void* scan_tmp;
  size_t scan_bytes;
};

__device__ __forceinline__ void record(int32_t* err, int code, int64_t tree, int64_t node) {
  if (atomicCAS(&err[0], 0, code) == 0) {
    err[1] = (int32_t)tree;
    err[2] = (int32_t)node;
  }
}

// Tree of global node gi: the last t with off[t] <= gi.
__device__ __forceinline__ int64_t tree_of(const DevEnsemble& e, int64_t gi) {
  int64_t lo = 0, hi = e.T - 1;
  while (lo < hi) {
    const int64_t mid = (lo + hi + 1) >> 1;
    if (e.off[mid] <= gi) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

__device__ __forceinline__ double cover_ratio(double child, double parent) {
  return parent > 0.0 ? child / parent : 0.0;
}

__device__ __forceinline__ bool is_leaf(const DevEnsemble& e, int64_t gi) {
  return e.left[gi] < 0 && e.right[gi] < 0;
}

__global__ void k_zero(double* p, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0.0;
}

__global__ void k_init(DevEnsemble e, Work w) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < e.N) {
    w.parent[i] = -1;
    w.npar[i] = 0;
    w.leaves[i] = 0;
    w.rank[i] = -1;
    w.merged[i] = 0;
  }
  if (i <= e.T) w.tree_leaves[i] = 0;
  if (i <= e.N) w.path_elems[i] = 0;
  if (i < 4) w.err[i] = 0;
}

// Tree table: offsets start at 0, grow strictly, end at N; groups in range.
__global__ void k_trees(DevEnsemble e, Work w) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= e.T) return;
  const int64_t a = e.off[t], b = e.off[t + 1];
  if ((t == 0 && a != 0) || b <= a || b - a > INT32_MAX || (t == e.T - 1 && b != e.N))
    record(w.err, kBadOffsets, t, -1);
  const int32_t g = e.group[t];
  if (g < 0 || g >= e.G) record(w.err, kBadGroup, t, -1);
}

// Per node: field checks and the parent links.
__global__ void k_nodes(DevEnsemble e, Work w) {
  const int64_t gi = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (gi >= e.N) return;
  const int64_t t = tree_of(e, gi);
  const int64_t base = e.off[t];
  const int64_t size = e.off[t + 1] - base;
  const int64_t n = gi - base;
  const double r = e.cover[gi];
  if (!(r >= 0.0) || !isfinite(r)) record(w.err, kBadCover, t, n);
  const int32_t a = e.left[gi], b = e.right[gi];
  if (a < 0 && b < 0) {
    if (!isfinite(e.value[gi])) record(w.err, kBadValue, t, n);
    return;
  }
  if (a < 0 || b < 0 || a >= size || b >= size) {
    record(w.err, kBadChild, t, n);
    return;
  }
  const int32_t d = e.feature[gi];
  if (d < 0 || d >= e.M) record(w.err, kBadFeature, t, n);
  if (isnan(e.threshold[gi])) record(w.err, kNanThreshold, t, n);
  atomicAdd(&w.npar[base + a], 1);
  atomicAdd(&w.npar[base + b], 1);
  w.parent[base + a] = (int32_t)n;
  w.parent[base + b] = (int32_t)n;
}

// Per node: every node has at most one parent, a root none.  Per reachable
// leaf: count it under every node on its way up.  A leaf whose way up does
// not end at its tree's root (a parentless inner node, or a loop found by
// taking more steps than the tree has nodes) is not part of the tree.
__global__ void k_count(DevEnsemble e, Work w) {
  const int64_t gi = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (gi >= e.N) return;
  const int64_t t = tree_of(e, gi);
  const int64_t base = e.off[t];
  const int64_t size = e.off[t + 1] - base;
  const int64_t n = gi - base;
  const int32_t np = w.npar[gi];
  if (np > 1) record(w.err, kTwoParents, t, n);
  if (n == 0 && np > 0) record(w.err, kRootHasParent, t, n);
  if (!is_leaf(e, gi)) return;
  int64_t steps = 0;
  int32_t a = (int32_t)n;
  while (a != 0) {
    a = w.parent[base + a];
    if (a < 0 || ++steps > size) return;  // not reachable from the root
  }
  if (steps > kMaxDepth) {
    record(w.err, kTooDeep, t, n);
    return;
  }
  a = (int32_t)n;
  atomicAdd(&w.leaves[base + a], 1);
  while (a != 0) {
    a = w.parent[base + a];
    atomicAdd(&w.leaves[base + a], 1);
  }
}

// The merged elements of the path ending at leaf n of the tree at base:
// features ascending with their ranges and zero fractions.  Returns the
// number of features, or -1 if more than kMaxMerged.
struct Merged {
  int32_t f[kMaxMerged];
  float lo[kMaxMerged];
  float hi[kMaxMerged];
  double z[kMaxMerged];
};

__device__ int merge_path(const DevEnsemble& e, const Work& w, int64_t base, int32_t n,
                          int32_t* chain, Merged& m) {
  // chain[0..d) = the path's nodes from the leaf's parent up to the root
  int d = 0;
  int32_t c = n;
  while (c != 0) {
    c = w.parent[base + c];
    chain[d++] = c;
  }
  int cnt = 0;
  for (int k = d - 1; k >= 0; --k) {
    const int32_t a = chain[k];
    const int32_t child = k > 0 ? chain[k - 1] : n;
    const int64_t ga = base + a;
    const int32_t f = e.feature[ga];
    const float th = e.threshold[ga];
    const bool right = e.right[ga] == child;
    const double ratio = cover_ratio(e.cover[base + child], e.cover[ga]);
    int i = 0;
    while (i < cnt && m.f[i] < f) ++i;
    if (i == cnt || m.f[i] != f) {
      if (cnt == kMaxMerged) return -1;
      for (int j = cnt; j > i; --j) {
        m.f[j] = m.f[j - 1];
        m.lo[j] = m.lo[j - 1];
        m.hi[j] = m.hi[j - 1];
        m.z[j] = m.z[j - 1];
      }
      m.f[i] = f;
      m.lo[i] = -INFINITY;
      m.hi[i] = INFINITY;
      m.z[i] = 1.0;
      ++cnt;
    }
    if (right) {
      if (th > m.lo[i]) m.lo[i] = th;
    } else {
      if (th < m.hi[i]) m.hi[i] = th;
    }
    m.z[i] = m.z[i] * ratio;
  }
  return cnt;
}

// Per reachable leaf: preorder rank (leaves under the left siblings passed on
// the way up) and merged length; reachable leaves per tree.
__global__ void k_rank(DevEnsemble e, Work w) {
  const int64_t gi = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (gi >= e.N) return;
  const int64_t t = tree_of(e, gi);
  const int64_t base = e.off[t];
  const int32_t n = (int32_t)(gi - base);
  if (n == 0) w.tree_leaves[t] = w.leaves[base];
  if (!is_leaf(e, gi) || w.leaves[gi] == 0) return;  // not reachable
  int32_t rank = 0;
  int32_t c = n;
  while (c != 0) {
    const int32_t a = w.parent[base + c];
    if (e.right[base + a] == c) rank += w.leaves[base + e.left[base + a]];
    c = a;
  }
  w.rank[gi] = rank;
  int32_t chain[kMaxDepth];
  Merged m;
  const int cnt = merge_path(e, w, base, n, chain, m);
  if (cnt < 0) {
    record(w.err, kTooLong, t, n);
    return;
  }
  w.merged[gi] = cnt;
}

// Per reachable leaf: its path index; elements per path.
__global__ void k_place(DevEnsemble e, Work w) {
  const int64_t gi = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (gi >= e.N) return;
  const int32_t r = w.rank[gi];
  if (r < 0) return;
  const int64_t t = tree_of(e, gi);
  const int64_t p = w.tree_off[t] + r;
  w.path_leaf[p] = gi;
  w.path_elems[p] = (int64_t)w.merged[gi] + 1;
}

// Per path: write its elements; its bias term v * prod(z).
__global__ void k_emit(DevEnsemble e, Work w, gts_path_element* __restrict__ out, int64_t P) {
  const int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= P) return;
  const int64_t gi = w.path_leaf[p];
  const int64_t t = tree_of(e, gi);
  const int64_t base = e.off[t];
  const int32_t g = e.group[t];
  int32_t chain[kMaxDepth];
  Merged m;
  const int cnt = merge_path(e, w, base, (int32_t)(gi - base), chain, m);
  const double v = e.value[gi];
  double prod = 1.0;
  for (int i = 0; i < cnt; ++i) prod = prod * m.z[i];
  w.term[p] = v * prod;
  if (out == nullptr) return;
  gts_path_element* el = out + w.elem_off[p];
  gts_path_element r;
  r.path_idx = p;
  r.feature_idx = -1;
  r.group = g;
  r.lower = -INFINITY;
  r.upper = INFINITY;
  r.zero_fraction = 1.0;
  r.v = v;
  el[0] = r;
  for (int i = 0; i < cnt; ++i) {
    r.feature_idx = m.f[i];
    r.lower = m.lo[i];
    r.upper = m.hi[i];
    r.zero_fraction = m.z[i];
    el[i + 1] = r;
  }
}

// Per tree: its paths' bias terms in path order.
__global__ void k_tree_sum(DevEnsemble e, Work w) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= e.T) return;
  double s = 0.0;
  for (int64_t p = w.tree_off[t]; p < w.tree_off[t + 1]; ++p) s = s + w.term[p];
  w.tree_sum[t] = s;
}

// Per group: its trees' sums in tree order.
__global__ void k_bias(DevEnsemble e, Work w, double* __restrict__ bias) {
  const int g = blockIdx.x * blockDim.x + threadIdx.x;
  if (g >= e.G) return;
  double s = 0.0;
  for (int64_t t = 0; t < e.T; ++t)
    if (e.group[t] == g) s = s + w.tree_sum[t];
  bias[g] = s;
}

// ---------------------------------------------------------------------------
// the model blob of a plan (gts_build_model_device)
// ---------------------------------------------------------------------------

// Features a plan's merged path may hold: plans are made only for models of
// at most 17 features.
constexpr int kPlanMaxM = 17;

// Arrays of the model blob being written.
template <typename Z>
struct BlobOut {
  int32_t* __restrict__ feat;
  float* __restrict__ lower;
  float* __restrict__ upper;
  Z* __restrict__ zero;
  int32_t* __restrict__ bin_start;
  int32_t* __restrict__ group_bins;
  Z* __restrict__ bias;
};

// Tree of every lane's path p, the last t with tree_paths[t] <= p (tree_paths
// is non-decreasing, tree_paths[0] = 0, tree_paths[T] = P).  The wave holds 64
// consecutive paths from p0 on.  It first narrows [0, T) to the tree of p0,
// probing 64 evenly spaced starts a round (two rounds for 4096 trees); then
// every lane counts, by bisection over the lanes, how many of the next 64 tree
// starts lie at or before its own path.  Only empty trees can put more than 63
// starts inside one wave; those lanes finish with a bisection of their own.
// Every lane of the wave must take part.
__device__ __forceinline__ int64_t wave_tree_of_path(const int32_t* __restrict__ tp, int64_t T,
                                                     int64_t p0, int64_t p) {
  const int lane = threadIdx.x & 63;
  int64_t lo = 0, n = T;   // the tree of p0 is in [lo, lo + n)
  while (n > 1) {
    const int64_t step = (n + 63) >> 6;
    const int64_t i = lo + lane * step;
    const uint64_t m = __ballot(i < lo + n && tp[i] <= p0);   // a prefix of the lanes, lane 0 in it
    const int64_t next = lo + (int64_t)(63 - __builtin_clzll(m)) * step;
    n = min(step, lo + n - next);
    lo = next;
  }
  const int64_t j = lo + 1 + lane;
  const int32_t v = j <= T ? tp[j] : INT32_MAX;   // non-decreasing over the lanes
  int c = 0;
  for (int b = 32; b >= 1; b >>= 1)
    if (__shfl(v, c + b - 1) <= p) c += b;
  if (c == 63 && __shfl(v, 63) <= p) c = 64;
  int64_t t = lo + c;
  if (c == 64) {
    int64_t hi = T - 1;
    while (t < hi) {
      const int64_t mid = (t + hi + 1) >> 1;
      if (tp[mid] <= p) t = mid;
      else hi = mid - 1;
    }
  }
  return min(t, T - 1);
}

// Per path: follow its turns from the root, merging the splits (ranges
// intersected, zero fractions multiplied in root-to-leaf order), then write
// the root (-1 - zero-fraction count, (-inf, +inf), v) and the features,
// those whose zero fraction is 0 in the blob's precision first, each group in
// ascending feature order, at the path's place; keep its bias term
// v * prod(z) (the product over the features in ascending order).  The merged
// ranges and fractions of the MF possible features stay in registers: every
// update goes through all MF slots with a select, since an array indexed by
// the split's feature would live in private memory.  A level issues one batch
// of loads, the node's own fields with its cover, whose ratio to the parent's
// cover is the fraction of the split above.
template <typename Z, int MF>
__global__ void k_build_paths(DevEnsemble e, const uint64_t* __restrict__ dirs,
                              const int32_t* __restrict__ dest,
                              const int32_t* __restrict__ tree_paths, int64_t P, int64_t E,
                              BlobOut<Z> out, double* __restrict__ term) {
  const int64_t wave0 = (int64_t)blockIdx.x * blockDim.x + (threadIdx.x & ~63);
  if (wave0 >= P) return;   // the whole wave
  const int64_t own = wave0 + (threadIdx.x & 63);
  const int64_t p = min(own, P - 1);
  const int64_t t = wave_tree_of_path(tree_paths, e.T, wave0, p);
  if (own >= P) return;
  const int64_t base = e.off[t];
  const int64_t size = e.off[t + 1] - base;
  if (size <= 0) return;   // never for an ensemble the plan walked
  float lo[MF], hi[MF];
  double z[MF];
#pragma unroll
  for (int k = 0; k < MF; ++k) {
    lo[k] = -INFINITY;
    hi[k] = INFINITY;
    z[k] = 1.0;
  }
  uint32_t on = 0;
  const uint64_t turns = dirs[p];
  int32_t node = 0;
  int32_t pf = -1;    // the feature of the split above node
  double pc = 0.0;    // the cover of node's parent
  for (int d = 0;; ++d) {
    const int64_t gi = base + node;
    const int32_t a = e.left[gi], b = e.right[gi], f = e.feature[gi];
    const float th = e.threshold[gi];
    const double c = e.cover[gi];
    if (pf >= 0) {
      const double r = cover_ratio(c, pc);
#pragma unroll
      for (int k = 0; k < MF; ++k) z[k] = k == pf ? z[k] * r : z[k];
    }
    if (a < 0 || b < 0 || d == 64) break;   // the leaf (or 64 turns taken)
    const bool right = (turns >> d) & 1ull;
    const int32_t child = right ? b : a;
    // never for an ensemble the plan walked
    if (child >= size || f < 0 || f >= MF) break;
    on |= 1u << f;
#pragma unroll
    for (int k = 0; k < MF; ++k) {
      lo[k] = k == f && right && th > lo[k] ? th : lo[k];
      hi[k] = k == f && !right && th < hi[k] ? th : hi[k];
    }
    pf = f;
    pc = c;
    node = child;
  }
  const double v = e.value[base + node];
  uint32_t zmask = 0;
  double prod = 1.0;
#pragma unroll
  for (int k = 0; k < MF; ++k) {
    const bool in = (on >> k) & 1u;
    zmask |= (uint32_t)(in && (Z)z[k] == Z(0)) << k;
    prod = in ? prod * z[k] : prod;
  }
  term[p] = v * prod;
  const int64_t d0 = dest[p];
  const int n0 = __builtin_popcount(zmask);
  // an ensemble other than the planned one could make the path longer than
  // its place: no write leaves the element arrays
  if (d0 < 0 || d0 + 1 + __builtin_popcount(on) > E) return;
  out.feat[d0] = -1 - n0;
  out.lower[d0] = -INFINITY;
  out.upper[d0] = INFINITY;
  out.zero[d0] = (Z)v;
  int64_t iz = d0 + 1, ir = d0 + 1 + n0;
#pragma unroll
  for (int k = 0; k < MF; ++k) {
    if ((on >> k) & 1u) {
      const bool zf = (zmask >> k) & 1u;
      const int64_t q = zf ? iz : ir;
      iz += zf ? 1 : 0;
      ir += zf ? 0 : 1;
      out.feat[q] = k;
      out.lower[q] = lo[k];
      out.upper[q] = hi[k];
      out.zero[q] = (Z)z[k];
    }
  }
}

// Lane l's value of x (l wave-uniform), through two scalar reads.
__device__ __forceinline__ double read_lane(double x, int l) {
  const long long bits = __double_as_longlong(x);
  const unsigned lo = (unsigned)__builtin_amdgcn_readlane((int)bits, l);
  const unsigned hi = (unsigned)__builtin_amdgcn_readlane((int)(bits >> 32), l);
  return __longlong_as_double((long long)(((unsigned long long)hi << 32) | lo));
}

// Sum of x[i] for i in [a, b) in index order, by one wave: the lanes load 64
// values at a time, then every lane adds them in order, reading each from
// its lane (all lanes hold the same sum).  sel[i] == want selects the values
// that take part (sel NULL: all).
__device__ __forceinline__ double wave_ordered_sum(const double* __restrict__ x, int64_t a,
                                                   int64_t b, const int32_t* __restrict__ sel,
                                                   int32_t want) {
  const int lane = threadIdx.x & 63;
  double s = 0.0;
  // the next chunk is loaded before the current one is added up, so the
  // loads wait behind the adds instead of the other way round
  int64_t i = a + lane;
  bool in = i < b && (sel == nullptr || sel[i] == want);
  double xi = in ? x[i] : 0.0;
  for (int64_t c = a; c < b; c += 64) {
    const uint64_t take0 = __ballot(in);
    const double cur = xi;
    i = c + 64 + lane;
    in = i < b && (sel == nullptr || sel[i] == want);
    xi = in ? x[i] : 0.0;
    if (take0 == ~0ull) {
#pragma unroll
      for (int l = 0; l < 64; ++l) s = s + read_lane(cur, l);
    } else {
#pragma unroll
      for (int l = 0; l < 64; ++l) {
        const double y = read_lane(cur, l);
        s = ((take0 >> l) & 1ull) ? s + y : s;
      }
    }
  }
  return s;
}

// Per tree (one wave): its paths' bias terms in path order.
__global__ void k_plan_tree_sums(const int32_t* __restrict__ tree_paths, int64_t T,
                                 const double* __restrict__ term, double* __restrict__ tree_sum) {
  const int64_t t = (int64_t)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
  if (t >= T) return;
  const double s = wave_ordered_sum(term, tree_paths[t], tree_paths[t + 1], nullptr, 0);
  if ((threadIdx.x & 63) == 0) tree_sum[t] = s;
}

// Per group (one wave): its trees' sums in tree order, in the blob's dtype.
template <typename Z>
__global__ void k_plan_bias(DevEnsemble e, const double* __restrict__ tree_sum, Z* __restrict__ bias) {
  const int64_t g = (int64_t)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
  if (g >= e.G) return;
  const double s = wave_ordered_sum(tree_sum, 0, e.T, e.group, (int32_t)g);
  if ((threadIdx.x & 63) == 0) bias[g] = (Z)s;
}

// The plan's bin starts and group ranges into the blob.
__global__ void k_plan_bins(const int32_t* __restrict__ bin_start, int64_t K,
                            const int32_t* __restrict__ group_bins, int64_t G,
                            int32_t* __restrict__ out_bins, int32_t* __restrict__ out_groups) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i <= K) out_bins[i] = bin_start[i];
  if (i <= G) out_groups[i] = group_bins[i];
}

// Zero bytes [a, b) of the blob, for up to kBlobArrays gaps (the padding that
// aligns every array); spans[2 j], spans[2 j + 1] is gap j.
struct Gaps {
  int64_t span[2 * kBlobArrays];
};

__global__ void k_zero_gaps(unsigned char* __restrict__ blob, Gaps gaps) {
  const int j = blockIdx.y;
  const int64_t a = gaps.span[2 * j], b = gaps.span[2 * j + 1];
  for (int64_t i = a + (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < b;
       i += (int64_t)gridDim.x * blockDim.x)
    blob[i] = 0;
}

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------

constexpr int64_t kAlign = 256;

inline int64_t up(int64_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

size_t scan_temp_bytes(int64_t n) {
  size_t bytes = 0;
  int64_t* null = nullptr;
  if (rocprim::exclusive_scan(nullptr, bytes, null, null, int64_t(0), (size_t)n,
                              rocprim::plus<int64_t>()) != hipSuccess)
    return 0;
  return bytes;
}

// Byte offsets of the workspace arrays; returns the total.
constexpr int kArrays = 15;

int64_t plan(int64_t T, int64_t N, int64_t* o, size_t* scan_bytes) {
  const int64_t n1 = N > 0 ? N : 1;
  *scan_bytes = std::max(scan_temp_bytes(T + 1), scan_temp_bytes(n1 + 1));
  const int64_t t1 = T > 0 ? T : 1;
  const int64_t sizes[kArrays] = {4 * 4,        0,            4 * n1,           4 * n1,
                                  4 * n1,       4 * n1,       4 * n1,           8 * (T + 1),
                                  8 * (T + 1),  8 * n1,       8 * (n1 + 1),     8 * (n1 + 1),
                                  8 * n1,       8 * t1,       (int64_t)*scan_bytes};
  int64_t at = 0;
  for (int i = 0; i < kArrays; ++i) {
    o[i] = at;
    at += up(sizes[i] > 0 ? sizes[i] : 1);
  }
  return at;
}

Work bind(void* ws, const int64_t* o, size_t scan_bytes) {
  char* b = static_cast<char*>(ws);
  Work w;
  w.err = reinterpret_cast<int32_t*>(b + o[0]);
  w.parent = reinterpret_cast<int32_t*>(b + o[2]);
  w.npar = reinterpret_cast<int32_t*>(b + o[3]);
  w.leaves = reinterpret_cast<int32_t*>(b + o[4]);
  w.rank = reinterpret_cast<int32_t*>(b + o[5]);
  w.merged = reinterpret_cast<int32_t*>(b + o[6]);
  w.tree_leaves = reinterpret_cast<int64_t*>(b + o[7]);
  w.tree_off = reinterpret_cast<int64_t*>(b + o[8]);
  w.path_leaf = reinterpret_cast<int64_t*>(b + o[9]);
  w.path_elems = reinterpret_cast<int64_t*>(b + o[10]);
  w.elem_off = reinterpret_cast<int64_t*>(b + o[11]);
  w.term = reinterpret_cast<double*>(b + o[12]);
  w.tree_sum = reinterpret_cast<double*>(b + o[13]);
  w.scan_tmp = b + o[14];
  w.scan_bytes = scan_bytes;
  return w;
}

const char* describe(int code) {
  switch (code) {
    case kBadOffsets: return "tree_node_offsets must start at 0, grow strictly and end at num_nodes";
    case kBadGroup: return "tree group outside [0, G)";
    case kBadCover: return "cover must be finite and >= 0";
    case kBadValue: return "leaf value is not finite";
    case kBadChild: return "child index out of range";
    case kBadFeature: return "split feature outside [0, M)";
    case kNanThreshold: return "threshold is NaN";
    case kTwoParents: return "node reached twice (shared child or cycle)";
    case kRootHasParent: return "the root is a child of another node (cycle)";
    case kTooDeep: return "path deeper than the device extraction supports (256 splits)";
    case kTooLong: return "merged path longer than a 64-element bin";
    default: return "malformed ensemble";
  }
}

inline unsigned blocks(int64_t n) { return (unsigned)std::max<int64_t>(1, (n + kThreads - 1) / kThreads); }

}  // namespace
}  // namespace gts

using namespace gts;

extern "C" gts_status gts_extract_workspace_bytes(int64_t num_trees, int64_t num_nodes,
                                                  int64_t* bytes) {
  clear_error();
  if (bytes == nullptr) return fail(GTS_EINVAL, "bytes must not be NULL");
  if (num_trees < 0 || num_nodes < 0) return fail(GTS_EINVAL, "sizes must be >= 0");
  int64_t o[kArrays];
  size_t sb = 0;
  *bytes = plan(num_trees, num_nodes, o, &sb);
  return GTS_OK;
}

namespace gts {
namespace {

gts_status extract_device(const gts_ensemble* ens, gts_path_element* d_out, int64_t capacity,
                          int64_t* num_elements, int64_t* num_paths, double* d_bias,
                          void* d_workspace, int64_t workspace_bytes, void* stream) {
  if (ens == nullptr || num_elements == nullptr || num_paths == nullptr)
    return fail(GTS_EINVAL, "ensemble, num_elements and num_paths must not be NULL");
  if (ens->num_features < 1 || ens->num_groups < 1 || ens->num_trees < 0 || ens->num_nodes < 0)
    return fail(GTS_EINVAL, "ensemble sizes out of range");
  if (capacity < 0) return fail(GTS_EINVAL, "capacity must be >= 0");
  if (d_out == nullptr && capacity > 0) return fail(GTS_EINVAL, "out is NULL but capacity > 0");
  const int64_t T = ens->num_trees, N = ens->num_nodes;
  if (T > INT32_MAX || N > INT32_MAX) return fail(GTS_EINVAL, "ensemble too large");
  *num_elements = 0;
  *num_paths = 0;
  if (T == 0) {
    if (N != 0) return fail(GTS_EINVAL, "num_nodes must be 0 without trees");
    if (d_bias) {
      hipLaunchKernelGGL(k_zero, dim3(blocks(ens->num_groups)), dim3(kThreads), 0,
                         static_cast<hipStream_t>(stream), d_bias, ens->num_groups);
      if (hipGetLastError() != hipSuccess) return fail(GTS_EDEVICE, "kernel launch failed");
    }
    return GTS_OK;
  }
  if (!ens->tree_node_offsets || !ens->tree_group || !ens->left || !ens->right ||
      !ens->feature || !ens->threshold || !ens->cover || !ens->value)
    return fail(GTS_EINVAL, "an ensemble array pointer is NULL");
  int64_t o[kArrays];
  size_t scan_bytes = 0;
  const int64_t need = plan(T, N, o, &scan_bytes);
  if (d_workspace == nullptr || workspace_bytes < need)
    return fail(GTS_EBUFSIZE, "workspace of %lld bytes needed", (long long)need);
  DevEnsemble e{ens->tree_node_offsets, ens->tree_group, ens->left, ens->right, ens->feature,
                ens->threshold, ens->cover, ens->value, T, N, ens->num_features,
                ens->num_groups};
  Work w = bind(d_workspace, o, scan_bytes);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const unsigned bn = blocks(std::max(N, T + 1)), bt = blocks(T);
  hipLaunchKernelGGL(k_init, dim3(bn), dim3(kThreads), 0, s, e, w);
  hipLaunchKernelGGL(k_trees, dim3(bt), dim3(kThreads), 0, s, e, w);
  if (hipGetLastError() != hipSuccess) return fail(GTS_EDEVICE, "kernel launch failed");
  // the node kernels read the offsets: check them first
  int32_t err[4] = {0, 0, 0, 0};
  if (hipMemcpyAsync(err, w.err, sizeof(err), hipMemcpyDeviceToHost, s) != hipSuccess ||
      hipStreamSynchronize(s) != hipSuccess)
    return fail(GTS_EDEVICE, "copy of the error word failed");
  if (err[0] != 0)
    return fail(GTS_EINVAL, "tree %d: %s", err[1], describe(err[0]));
  const unsigned b = blocks(N);
  hipLaunchKernelGGL(k_nodes, dim3(b), dim3(kThreads), 0, s, e, w);
  hipLaunchKernelGGL(k_count, dim3(b), dim3(kThreads), 0, s, e, w);
  hipLaunchKernelGGL(k_rank, dim3(b), dim3(kThreads), 0, s, e, w);
  if (hipGetLastError() != hipSuccess) return fail(GTS_EDEVICE, "kernel launch failed");
  size_t sb = w.scan_bytes;
  if (rocprim::exclusive_scan(w.scan_tmp, sb, w.tree_leaves, w.tree_off, int64_t(0),
                              (size_t)(T + 1), rocprim::plus<int64_t>(), s) != hipSuccess)
    return fail(GTS_EDEVICE, "scan over trees failed");
  hipLaunchKernelGGL(k_place, dim3(b), dim3(kThreads), 0, s, e, w);
  int64_t P = 0;
  if (hipMemcpyAsync(err, w.err, sizeof(err), hipMemcpyDeviceToHost, s) != hipSuccess ||
      hipMemcpyAsync(&P, w.tree_off + T, sizeof(P), hipMemcpyDeviceToHost, s) != hipSuccess ||
      hipStreamSynchronize(s) != hipSuccess)
    return fail(GTS_EDEVICE, "copy of the path count failed");
  if (err[0] != 0)
    return fail(err[0] == kTooLong ? GTS_EPATHLEN : GTS_EINVAL, "tree %d node %d: %s", err[1],
                err[2], describe(err[0]));
  // path_elems[P] is 0 (k_init), so the scan's last entry is the total
  sb = w.scan_bytes;
  if (rocprim::exclusive_scan(w.scan_tmp, sb, w.path_elems, w.elem_off, int64_t(0),
                              (size_t)(P + 1), rocprim::plus<int64_t>(), s) != hipSuccess)
    return fail(GTS_EDEVICE, "scan over paths failed");
  int64_t n = 0;
  if (hipMemcpyAsync(&n, w.elem_off + P, sizeof(n), hipMemcpyDeviceToHost, s) != hipSuccess ||
      hipStreamSynchronize(s) != hipSuccess)
    return fail(GTS_EDEVICE, "copy of the element count failed");
  *num_paths = P;
  *num_elements = n;
  if (d_out != nullptr && n > capacity)
    return fail(GTS_EBUFSIZE, "capacity %lld < %lld elements", (long long)capacity,
                (long long)n);
  if (d_out == nullptr && d_bias == nullptr) return GTS_OK;
  hipLaunchKernelGGL(k_emit, dim3(blocks(P)), dim3(kThreads), 0, s, e, w, d_out, P);
  if (d_bias) {
    hipLaunchKernelGGL(k_tree_sum, dim3(bt), dim3(kThreads), 0, s, e, w);
    hipLaunchKernelGGL(k_bias, dim3(blocks(ens->num_groups)), dim3(kThreads), 0, s, e, w, d_bias);
  }
  if (hipGetLastError() != hipSuccess) return fail(GTS_EDEVICE, "kernel launch failed");
  return GTS_OK;
}

}  // namespace
}  // namespace gts

extern "C" gts_status gts_extract_paths_device(const gts_ensemble* ens, gts_path_element* d_out,
                                               int64_t capacity, int64_t* num_elements,
                                               int64_t* num_paths, double* d_bias,
                                               void* d_workspace, int64_t workspace_bytes,
                                               void* stream) {
  clear_error();
  return extract_device(ens, d_out, capacity, num_elements, num_paths, d_bias, d_workspace,
                        workspace_bytes, stream);
}

// ---------------------------------------------------------------------------
// gts_build_model_device
// ---------------------------------------------------------------------------

namespace gts {
namespace {

// Workspace of gts_build_model_device: path terms [P], tree sums [T].
int64_t build_workspace(const gts_plan* plan, int64_t* tree_off) {
  const int64_t a = up(8 * std::max<int64_t>(1, plan->num_paths));
  *tree_off = a;
  return a + up(8 * std::max<int64_t>(1, plan->num_trees));
}

template <typename Z>
gts_status build_device(const gts_ensemble* ens, const gts_model* m, const gts_plan* plan,
                        const char* d_plan, char* d_model, char* ws, hipStream_t s) {
  DevEnsemble e{ens->tree_node_offsets, ens->tree_group, ens->left, ens->right, ens->feature,
                ens->threshold, ens->cover, ens->value, ens->num_trees, ens->num_nodes,
                ens->num_features, ens->num_groups};
  const int64_t P = plan->num_paths, T = plan->num_trees, K = plan->num_bins;
  const int64_t G = ens->num_groups;
  BlobOut<Z> out{reinterpret_cast<int32_t*>(d_model + m->off[kFeat]),
                 reinterpret_cast<float*>(d_model + m->off[kLower]),
                 reinterpret_cast<float*>(d_model + m->off[kUpper]),
                 reinterpret_cast<Z*>(d_model + m->off[kZero]),
                 reinterpret_cast<int32_t*>(d_model + m->off[kBinStart]),
                 reinterpret_cast<int32_t*>(d_model + m->off[kGroupBins]),
                 reinterpret_cast<Z*>(d_model + m->off[kBias])};
  const uint64_t* dirs = reinterpret_cast<const uint64_t*>(d_plan + plan->off[0]);
  const int32_t* dest = reinterpret_cast<const int32_t*>(d_plan + plan->off[1]);
  const int32_t* tree_paths = reinterpret_cast<const int32_t*>(d_plan + plan->off[2]);
  const int32_t* bins = reinterpret_cast<const int32_t*>(d_plan + plan->off[3]);
  const int32_t* groups = reinterpret_cast<const int32_t*>(d_plan + plan->off[4]);
  int64_t tree_off = 0;
  build_workspace(plan, &tree_off);
  double* term = reinterpret_cast<double*>(ws);
  double* tree_sum = reinterpret_cast<double*>(ws + tree_off);
  // the alignment padding after every array
  const size_t zb = sizeof(Z);
  const int64_t sizes[kBlobArrays] = {4 * m->num_elements, 4 * m->num_elements,
                                      4 * m->num_elements, (int64_t)zb * m->num_elements,
                                      4 * (K + 1),         4 * (G + 1),
                                      (int64_t)zb * G};
  Gaps gaps;
  for (int k = 0; k < kBlobArrays; ++k) {
    gaps.span[2 * k] = m->off[k] + sizes[k];
    gaps.span[2 * k + 1] = k + 1 < kBlobArrays ? m->off[k + 1] : m->bytes;
  }
  hipLaunchKernelGGL(k_zero_gaps, dim3(1, kBlobArrays), dim3(kThreads), 0, s,
                     reinterpret_cast<unsigned char*>(d_model), gaps);
  // a model of at most 8 features carries 8 slots per path, any other 17
  if (P > 0 && e.M <= 8)
    hipLaunchKernelGGL((k_build_paths<Z, 8>), dim3(blocks(P)), dim3(kThreads), 0, s, e, dirs,
                       dest, tree_paths, P, m->num_elements, out, term);
  else if (P > 0)
    hipLaunchKernelGGL((k_build_paths<Z, kPlanMaxM>), dim3(blocks(P)), dim3(kThreads), 0, s, e,
                       dirs, dest, tree_paths, P, m->num_elements, out, term);
  hipLaunchKernelGGL(k_plan_bins, dim3(blocks(std::max(K, G) + 1)), dim3(kThreads), 0, s, bins,
                     K, groups, G, out.bin_start, out.group_bins);
  constexpr int kWaves = kThreads / 64;
  if (T > 0)
    hipLaunchKernelGGL(k_plan_tree_sums, dim3((unsigned)((T + kWaves - 1) / kWaves)),
                       dim3(kThreads), 0, s, tree_paths, T, term, tree_sum);
  hipLaunchKernelGGL(k_plan_bias<Z>, dim3((unsigned)((G + kWaves - 1) / kWaves)),
                     dim3(kThreads), 0, s, e, tree_sum, out.bias);
  const hipError_t err = hipGetLastError();
  if (err != hipSuccess) return fail(GTS_EDEVICE, "kernel launch failed: %s", hipGetErrorString(err));
  return GTS_OK;
}

}  // namespace
}  // namespace gts

extern "C" gts_status gts_build_workspace_bytes(const gts_plan* plan, int64_t* bytes) {
  clear_error();
  if (plan == nullptr || bytes == nullptr) return fail(GTS_EINVAL, "plan and bytes must not be NULL");
  int64_t t = 0;
  *bytes = build_workspace(plan, &t);
  return GTS_OK;
}

extern "C" gts_status gts_build_model_device(const gts_ensemble* ens, const gts_model* model,
                                             const gts_plan* plan, const void* d_plan,
                                             void* d_model, void* d_workspace,
                                             int64_t workspace_bytes, void* stream) {
  clear_error();
  if (ens == nullptr || model == nullptr || plan == nullptr || d_plan == nullptr ||
      d_model == nullptr || d_workspace == nullptr)
    return fail(GTS_EINVAL, "NULL argument");
  gts_status st = check_model(model);
  if (st != GTS_OK) return st;
  if (model->flags & GTS_MODEL_PRUNED) return fail(GTS_EINVAL, "a pruned model has no plan");
  if (ens->num_trees != plan->num_trees || ens->num_nodes != plan->num_nodes ||
      model->num_paths != plan->num_paths || model->num_bins != plan->num_bins ||
      ens->num_features != model->num_features || ens->num_groups != model->num_groups)
    return fail(GTS_EINVAL, "the ensemble, model and plan do not belong together");
  if (ens->num_features > kPlanMaxM) return fail(GTS_EINVAL, "a plan needs M <= %d", kPlanMaxM);
  if (plan->num_trees > 0 &&
      (!ens->tree_node_offsets || !ens->tree_group || !ens->left || !ens->right ||
       !ens->feature || !ens->threshold || !ens->cover || !ens->value))
    return fail(GTS_EINVAL, "an ensemble array pointer is NULL");
  int64_t t = 0;
  const int64_t need = build_workspace(plan, &t);
  if (workspace_bytes < need)
    return fail(GTS_EBUFSIZE, "workspace of %lld bytes needed", (long long)need);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const char* dp = static_cast<const char*>(d_plan);
  char* dm = static_cast<char*>(d_model);
  char* ws = static_cast<char*>(d_workspace);
  return model->dtype == GTS_F64 ? build_device<double>(ens, model, plan, dp, dm, ws, s)
                                 : build_device<float>(ens, model, plan, dp, dm, ws, s);
}

// ---------------------------------------------------------------------------
// allocation-free variant: the workspace is a fixed device array
// ---------------------------------------------------------------------------

// Workspace of gts_extract_paths_device_noalloc on every device the library
// runs on (each device holds its own copy, from module load to process exit).
// Host code never uses this name as an address: the device address comes
// from hipGetSymbolAddress, once per device.
static __device__ __align__(256) unsigned char scratch[GTS_EXTRACT_NOALLOC_BYTES];

namespace gts {
namespace {

// The device address of `scratch` on the current device, looked up on the
// first call on that device (with it current) and kept.
gts_status scratch_address(void** out) {
  static std::mutex mu;
  static std::vector<void*> addr;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return fail(GTS_EDEVICE, "no HIP device");
  std::lock_guard<std::mutex> lock(mu);
  if ((int)addr.size() <= dev) addr.resize((size_t)dev + 1, nullptr);
  if (addr[(size_t)dev] == nullptr) {
    void* p = nullptr;
    const hipError_t err = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (err != hipSuccess || p == nullptr)
      return fail(GTS_EDEVICE, "hipGetSymbolAddress of the extraction workspace failed: %s",
                  hipGetErrorString(err));
    addr[(size_t)dev] = p;
  }
  *out = addr[(size_t)dev];
  return GTS_OK;
}

}  // namespace
}  // namespace gts

extern "C" gts_status gts_extract_paths_device_noalloc(const gts_ensemble* ens,
                                                       gts_path_element* d_out, int64_t capacity,
                                                       int64_t* num_elements, int64_t* num_paths,
                                                       double* d_bias, void* stream) {
  clear_error();
  if (ens == nullptr) return fail(GTS_EINVAL, "ensemble must not be NULL");
  if (ens->num_trees < 0 || ens->num_nodes < 0)
    return fail(GTS_EINVAL, "ensemble sizes out of range");
  int64_t o[kArrays];
  size_t scan_bytes = 0;
  const int64_t need = plan(ens->num_trees, ens->num_nodes, o, &scan_bytes);
  if (need > GTS_EXTRACT_NOALLOC_BYTES)
    return fail(GTS_EINVAL,
                "ensemble of %lld trees and %lld nodes needs %lld bytes of workspace; "
                "gts_extract_paths_device_noalloc holds %lld (use gts_extract_paths_device)",
                (long long)ens->num_trees, (long long)ens->num_nodes, (long long)need,
                (long long)GTS_EXTRACT_NOALLOC_BYTES);
  void* ws = nullptr;
  const gts_status st = scratch_address(&ws);
  if (st != GTS_OK) return st;
  return extract_device(ens, d_out, capacity, num_elements, num_paths, d_bias, ws,
                        GTS_EXTRACT_NOALLOC_BYTES, stream);
}
