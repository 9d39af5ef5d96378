// SHAP and SHAP-interaction kernels of libgts for gfx950 (CDNA4, wave64),
// included by the translation units that instantiate them
// (gts_shap_f32.hip, gts_shap_f64.hip, gts_inter_f32.hip, gts_inter_f64.hip).
//
// Work units.  The model arrives packed into bins of at most 64 path
// elements (Section 3.3, Best-Fit-Decreasing).  A wave takes one bin at a
// time and loads it with one element per lane -- the element-per-thread layout
// of the paper's kernel -- prefetching the next bin while it computes.  It
// copies the bin into a per-wave staging area in LDS, and a ballot over "is a
// root element" gives the lane where each path starts.
//
// Lanes.  Unlike the paper's kernel, a lane does not own a path element: it
// owns a (row, path) pair and runs the whole per-path dynamic programme of
// Algorithm 1 in its registers.  A wave covers RW rows x (64/RW) paths.  With
// RW == 64 all lanes share one path and read its elements from the staging
// area at the same address (an LDS broadcast); with fewer rows per wave each
// group of RW lanes reads its own path's elements.  Trip counts are
// compile-time constants (one variant per path length up to 16 features, 8
// for interactions), so a wave never diverges on path length.  This does the
// q^2 work of a path once per row instead of spreading it over q lanes that
// then need q shuffles each.  Each kernel is built for the model's longest
// path: up to 8 features, up to 12, up to 16 (fp64 arithmetic), or longer;
// only the last holds the runtime-loop code for long paths and its per-lane
// private arrays.
//
// Dead pairs.  An element whose zero fraction is 0 gives the factor
// z + o t = 0 for every row outside its range, so such a (row, path) has all
// weights 0 and contributes exactly nothing (the zero-cover pruning of
// Algorithm 1).  The host stores those elements first in their path and their
// count in the root.  With one path per wave (RW == 64) a wave skips every
// path that no row of its tile reaches: for models of at most 16 features it
// finds them for a whole bin at once, before staging it, from rank tables of
// the tile's row keys; otherwise it tests each path's elements in turn.  The
// multi-path rounds (RW < 64) compute every pair.
//
// Arithmetic.  EXTEND keeps permutation weights w_k, which are the
// coefficients E_k of prod_k (z_k + o_k t) scaled by k!(l-k)!/(l+1)!.  The
// kernels keep E_k: adding an element is E_k <- z E_k + o E_{k-1} (one
// multiply-add), and the scale factors reappear in the final sums as the
// Shapley weights c_k = k!(q-1-k)!/q!.  UNWIND of an element with o = 1
// divides the polynomial by (z + t) from the top coefficient down, like
// Algorithm 1's o != 0 branch.  Its Shapley-weighted sum is linear in the
// quotient, so it is a polynomial in -z whose coefficients
// G_m = sum_{j>m} c_{j-1-m} E_j are shared by every element of the path: one
// multiply-add per coefficient per element (Horner) instead of a division and
// a weighted sum.  For o = 0 the contribution reduces to -v * sum_k c_k E_k,
// shared by every such element, so no division by a zero fraction is ever
// needed.  Per-element constants of a path (v (1 - z)) are computed once per
// bin when it is staged, not once per row.
//
// Accumulation.  A workgroup owns a tile of RW rows of one output group and a
// slice of that group's bins.  Contributions go to a phi tile in LDS (an
// atomic add built from compare-and-swap, the compare-and-swaps of a path
// issued together so their LDS round trips overlap) or, when a wave has a
// tile of its own and one path at a time, a plain read-modify-write.  An
// interaction pair is added to one of its two entries and the tile write sums
// the mirror entries, so the output is exactly symmetric.  The tile is written
// to HBM once (atomically added when several workgroups share the row tile).
#pragma once

#include <hip/hip_runtime.h>

#include <algorithm>
#include <climits>
#include <cstdint>
#include <type_traits>

#include "gts_internal.h"
#include "gts_launch.h"

namespace gts {
namespace {

constexpr int kPastEnd = INT_MIN;   // feature slot of a lane past the end of its bin

// Ordered key of a float: for non-NaN a and b, a < b exactly when
// fkey(a) < fkey(b) as signed integers (-0 is taken as +0 first, so equal
// floats get equal keys).  The range test lower <= x < upper becomes
// (unsigned)(fkey(x) - klo) < span with klo = fkey(lower) and
// span = max(fkey(upper) - klo, 0): one unsigned compare, exact for every
// non-NaN x and empty (lower >= upper) ranges, and false for a NaN x (its key
// lies outside [fkey(-inf), fkey(+inf)]).
__device__ __forceinline__ int fkey(float x) {
  const int i = __float_as_int(x + 0.0f);
  return i ^ ((i >> 31) & 0x7fffffff);
}
__device__ __forceinline__ unsigned key_span(int klo, int khi) {
  return khi > klo ? (unsigned)khi - (unsigned)klo : 0u;
}
__device__ __forceinline__ bool in_range(int kx, int klo, unsigned span) {
  return (unsigned)kx - (unsigned)klo < span;
}

// The interaction tile of a row keeps the upper triangle of the symmetric
// (M+1) x (M+1) block, row by row: entry (a, b), a <= b, at tri_row(a) + b
// with tri_row(a) = a W - a (a + 1) / 2 (W = M + 1 entries per full row).
__device__ __forceinline__ int tri_row(int a, int W) { return a * W - ((a * (a + 1)) >> 1); }
__device__ __forceinline__ int tri_at(int a, int b, int W) {
  return a <= b ? tri_row(a, W) + b : tri_row(b, W) + a;
}

template <typename T>
struct DevModel {
  const int32_t* __restrict__ feat;
  const float* __restrict__ lower;
  const float* __restrict__ upper;
  const T* __restrict__ zero;         // zero fraction; leaf value on root elements
  const int32_t* __restrict__ bin_start;
  const int32_t* __restrict__ group_bins;
  const T* __restrict__ bias;
  int32_t M;
  int32_t G;
};

template <typename T>
DevModel<T> dev_model(const gts_model* m, const void* blob) {
  const char* b = static_cast<const char*>(blob);
  DevModel<T> d;
  d.feat = reinterpret_cast<const int32_t*>(b + m->off[kFeat]);
  d.lower = reinterpret_cast<const float*>(b + m->off[kLower]);
  d.upper = reinterpret_cast<const float*>(b + m->off[kUpper]);
  d.zero = reinterpret_cast<const T*>(b + m->off[kZero]);
  d.bin_start = reinterpret_cast<const int32_t*>(b + m->off[kBinStart]);
  d.group_bins = reinterpret_cast<const int32_t*>(b + m->off[kGroupBins]);
  d.bias = reinterpret_cast<const T*>(b + m->off[kBias]);
  d.M = m->num_features;
  d.G = m->num_groups;
  return d;
}

struct Launch {
  int64_t rows;
  int64_t ld;
  int32_t tiles;     // row tiles
  int32_t splits;    // bin slices per group
  int32_t sx;        // LDS row stride of the X tile (floats)
  int32_t sp;        // LDS row stride of the phi tile (elements; interactions:
                     // the upper triangle, W (W + 1) / 2 entries)
  int32_t width;     // phi entries per (row, group): M+1 or (M+1)^2
  int32_t accumulate;  // 1: atomically add the tile to phi (phi pre-zeroed)
  int32_t sorted;      // 1: inside a bin, paths never grow in length
  int32_t rank_off;    // LDS offset of the rank tables; 0: none
  // A pruned model's bin count is known only on the device: its workgroups
  // use min(splits, max(min_splits, bins / (32 waves))) slices, rounded down
  // to a multiple of split_step, and the others return at once (adaptive).
  int32_t adaptive;
  int32_t min_splits;
  int32_t split_step;
};

// Makes v a value the compiler must hold in registers at this point, so the
// code that computes it stays on every lane's path: a select between it and
// another value then costs one v_cndmask instead of a divergent branch around
// its computation.
template <typename T>
__device__ __forceinline__ void keep(T& v) {
  asm volatile("" : "+v"(v));
}

// Shapley weight of a coalition of size k among the other n-1 players:
// k! (n-1-k)! / n!  =  1 / (n * C(n-1, k)).
__host__ __device__ constexpr double shapley_weight(int n, int k) {
  double c = 1.0;
  for (int i = 1; i <= k; ++i) c = c * (double)(n - i) / (double)i;
  return 1.0 / ((double)n * c);
}

// Add to a phi-tile entry in LDS.  A compare-and-swap loop on the bit
// pattern: gfx950 executes the LDS float add atomic (ds_add_f32) one lane at
// a time, about 190 cycles per wave64 instruction, while the integer
// compare-and-swap runs at the rate of a plain read-modify-write; without a
// conflict the loop runs once.
__device__ __forceinline__ void lds_add(float* p, float v) {
  unsigned* q = reinterpret_cast<unsigned*>(p);
  unsigned old = *q, assumed;
  do {
    assumed = old;
    old = atomicCAS(q, assumed, __float_as_uint(__uint_as_float(assumed) + v));
  } while (old != assumed);
}
__device__ __forceinline__ void lds_add(double* p, double v) {
  unsigned long long* q = reinterpret_cast<unsigned long long*>(p);
  unsigned long long old = *q, assumed;
  do {
    assumed = old;
    old = atomicCAS(q, assumed,
                    (unsigned long long)__double_as_longlong(__longlong_as_double((long long)assumed) + v));
  } while (old != assumed);
}

// Bit patterns of the tile entries, for compare-and-swap.
template <typename T> struct Bits;
template <> struct Bits<float> {
  using U = unsigned;
  static __device__ __forceinline__ U of(float x) { return __float_as_uint(x); }
  static __device__ __forceinline__ float val(U u) { return __uint_as_float(u); }
};
template <> struct Bits<double> {
  using U = unsigned long long;
  static __device__ __forceinline__ U of(double x) { return (U)__double_as_longlong(x); }
  static __device__ __forceinline__ double val(U u) { return __longlong_as_double((long long)u); }
};

// How a lane adds the contributions of one path to the phi tile.
//   kExclusive  no other lane or wave updates these entries meanwhile (a
//               wave-private tile with one path per wave): plain
//               read-modify-writes, all reads issued before any write.
//   kBatched    all reads are issued, then all compare-and-swaps, so the LDS
//               round trips overlap.  For one path per wave, or entries that
//               rarely coincide across lanes (interaction pairs).
//   kPaired     read and compare-and-swap entry by entry; the check of the
//               results waits until the end.  For several paths per wave:
//               two of its paths may share a feature, but rarely at the same
//               step.
// An entry that another lane or wave changed between the read and the
// compare-and-swap is added again with the compare-and-swap loop.
enum AddMode { kExclusive, kBatched, kPaired };

// Add val[i] to *p[i] for every i with on[i]; the addresses of one lane are
// distinct.  p[i] must be a valid tile address even where on[i] is false.
template <AddMode MODE, typename T, int N>
__device__ __forceinline__ void tile_add(T* const (&p)[N], const T (&val)[N], const bool (&on)[N]) {
  if constexpr (MODE == kExclusive) {
    T old[N];
#pragma unroll
    for (int i = 0; i < N; ++i) old[i] = *p[i];
#pragma unroll
    for (int i = 0; i < N; ++i)
      if (on[i]) *p[i] = old[i] + val[i];
  } else {
    using U = typename Bits<T>::U;
    U old[N], got[N];
    if constexpr (MODE == kBatched) {
#pragma unroll
      for (int i = 0; i < N; ++i) old[i] = *reinterpret_cast<const U*>(p[i]);
#pragma unroll
      for (int i = 0; i < N; ++i)
        got[i] = on[i] ? atomicCAS(reinterpret_cast<U*>(p[i]), old[i],
                                   Bits<T>::of(Bits<T>::val(old[i]) + val[i]))
                       : old[i];
    } else {
      // every lane swaps, so no lane branches around its swap: an entry that
      // is off adds -0.0, which leaves every value as it is (-0.0 included)
#pragma unroll
      for (int i = 0; i < N; ++i) {
        const T add = on[i] ? val[i] : T(-0.0);
        old[i] = *reinterpret_cast<const U*>(p[i]);
        got[i] = atomicCAS(reinterpret_cast<U*>(p[i]), old[i],
                           Bits<T>::of(Bits<T>::val(old[i]) + add));
      }
    }
    bool retry = false;
#pragma unroll
    for (int i = 0; i < N; ++i) retry |= got[i] != old[i];
    if (retry) {
#pragma unroll
      for (int i = 0; i < N; ++i)
        if (got[i] != old[i]) lds_add(p[i], on[i] ? val[i] : T(-0.0));
    }
  }
}

// Single entry, for the runtime-length path code.
template <bool EXCL, typename T>
__device__ __forceinline__ void acc_add(T* p, T v) {
  if constexpr (EXCL) *p += v;
  else lds_add(p, v);
}

// One bin, one element per lane.
template <typename T>
struct Bin {
  int feat;   // feature; on a root -1 - n0; kPastEnd past the end of the bin
  int klo;    // range [lower, upper) as fkey(lower) and the key span
  unsigned span;
  T z;        // zero fraction, or the leaf value on a root
  int len;    // elements in the bin (uniform)
};

template <typename T>
__device__ __forceinline__ Bin<T> load_bin(const DevModel<T>& d, int bi, int lane) {
  Bin<T> b;
  const int e0 = d.bin_start[bi];
  b.len = d.bin_start[bi + 1] - e0;
  if (lane < b.len) {
    const int e = e0 + lane;
    b.feat = d.feat[e];
    b.klo = fkey(d.lower[e]);
    b.span = key_span(b.klo, fkey(d.upper[e]));
    b.z = d.zero[e];
  } else {
    b.feat = kPastEnd;
    b.klo = 0;
    b.span = 0u;
    b.z = T(0);
  }
  return b;
}

// One wave's copy of its current bin in LDS.  head[slot] = (feature, fkey of
// lower, key span of the range, fp32 z bits); aux[slot] holds w = v (1 - z), v the leaf
// value of the element's path (and z itself for fp64 models); on a root, z
// and w hold v.  path[t] = slot of the t-th root | (features of its path) << 8
// | (its zero-fraction elements) << 16.
//
// GAPPED (several paths per wave): element e of the bin sits in slot
// e + (number of even-length paths before its path).  The gap after every
// path of even length makes the distance between consecutive path starts
// odd, so lanes reading the k-th elements of up to 8 paths of equal length at
// once hit different LDS banks.  Slot kSlots holds a neutral
// element (feature 0, range (-inf, +inf), z = 1, w = 0): a player present
// and absent alike, which changes no other player's Shapley value.  A lane
// whose path is shorter than the wave's longest reads it in place of the
// elements past its path's end.  Without GAPPED (one path per wave, every
// read a broadcast) element e sits in slot e.
template <typename T> struct Aux;   // fp64 models; fp32 models keep w alone
template <> struct alignas(16) Aux<double> {
  double z, w;
};

template <typename T, bool GAPPED>
struct Stage {
  static constexpr int kSlots = GAPPED ? 96 : 64;   // 64 elements + a gap per even-length path
  using AuxT = std::conditional_t<sizeof(T) == 4, float, Aux<T>>;
  int4 head[kSlots + 1];
  AuxT aux[kSlots + 1];
  int path[64];

  __device__ __forceinline__ T w(int e) const {
    if constexpr (std::is_same_v<AuxT, float>) return aux[e];
    else return aux[e].w;
  }
  __device__ __forceinline__ T z(int e) const {
    if constexpr (sizeof(T) == 4) return __int_as_float(head[e].w);
    else return aux[e].z;
  }
};

template <typename T, bool GAPPED>
__device__ __forceinline__ void init_stage(Stage<T, GAPPED>* st, int lane) {
  using S = Stage<T, GAPPED>;
  if (lane == 0) {
    const int klo = fkey(-INFINITY);
    st->head[S::kSlots] = make_int4(0, klo, (int)key_span(klo, fkey(INFINITY)),
                                    __float_as_int(1.0f));
    typename S::AuxT n{};
    if constexpr (std::is_same_v<typename S::AuxT, float>) {
      n = 0.0f;
    } else {
      if constexpr (sizeof(T) == 8) n.z = 1.0;
      n.w = T(0);
    }
    st->aux[S::kSlots] = n;
  }
}

// Where the paths of a bin start: roots = the lanes of its root elements,
// rl = this lane's root, len = on a root lane, the path's elements, n0 = on
// a root lane, its zero-fraction elements (stored first), info = (len - 1) |
// (n0 << 8).
struct BinIndex {
  uint64_t roots;
  int rl, len, n0, info;
  bool root;
};

template <typename T>
__device__ __forceinline__ BinIndex index_bin(const Bin<T>& b, int lane) {
  BinIndex ix;
  ix.root = lane < b.len && b.feat < 0;
  ix.n0 = ix.root ? -1 - b.feat : 0;
  ix.roots = __ballot(ix.root);
  const uint64_t upto = ix.roots & ((2ull << lane) - 1ull);      // roots at or below this lane
  ix.rl = upto ? 63 - __clzll((long long)upto) : lane;
  const uint64_t above = ix.roots & ~((2ull << lane) - 1ull);
  ix.len = (above ? __builtin_ctzll(above) : b.len) - lane;
  ix.info = (ix.len - 1) | (ix.n0 << 8);
  return ix;
}

// Stages a bin (indexed by index_bin); returns its number of paths.  On a
// root lane, info holds the path's features | its zero-fraction elements << 8.
template <typename T, bool GAPPED>
__device__ __forceinline__ int stage_bin(Stage<T, GAPPED>* st, const Bin<T>& b, int lane,
                                         const BinIndex& ix) {
  int slot = lane;
  if constexpr (GAPPED) {
    const uint64_t evens = __ballot(ix.root && (ix.len & 1) == 0);
    slot += __popcll(evens & ((1ull << ix.rl) - 1ull));
  }
  const T v = __shfl(b.z, ix.rl);   // a root's zero-fraction slot holds v
  const T w = ix.root ? v : v * (T(1) - b.z);
  st->head[slot] = make_int4(b.feat, b.klo, (int)b.span,
                             sizeof(T) == 4 ? __float_as_int((float)b.z) : 0);
  typename Stage<T, GAPPED>::AuxT ax{};
  if constexpr (std::is_same_v<typename Stage<T, GAPPED>::AuxT, float>) {
    ax = w;
  } else {
    if constexpr (sizeof(T) == 8) ax.z = b.z;
    ax.w = w;
  }
  st->aux[slot] = ax;
  const int rank = __builtin_amdgcn_mbcnt_hi((unsigned)(ix.roots >> 32),
                                             __builtin_amdgcn_mbcnt_lo((unsigned)ix.roots, 0u));
  if (ix.root) st->path[rank] = slot | (ix.info << 8);
  // the stores above are read by other lanes of this wave only
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  return __popcll(ix.roots);
}

// Fields of a staged path word.
__device__ __forceinline__ int path_slot(int info) { return info & 0xff; }
__device__ __forceinline__ int path_q(int info) { return (info >> 8) & 0xff; }
__device__ __forceinline__ int path_n0(int info) { return info >> 16; }

// Feature, presence test o_k = [lower <= x < upper] (on keys), zero fraction and
// v (1 - z) of the first Q feature elements of the path whose root is in
// slot s (wave-uniform when UNIFORM).  A lane whose path has q < Q features
// reads the neutral element for k >= q; on[k] = k < q marks the elements
// whose contributions are written.
template <typename T, int Q, bool UNIFORM, bool GAPPED>
__device__ __forceinline__ void load_path(const Stage<T, GAPPED>* st, int s, int q,
                                          const int* __restrict__ xrow, int (&f)[Q],
                                          bool (&o)[Q], T (&z)[Q], T (&w)[Q], bool (&on)[Q]) {
#pragma unroll
  for (int k = 0; k < Q; ++k) {
    const bool real = UNIFORM || k < q;
    const int e = real ? s + 1 + k : Stage<T, GAPPED>::kSlots;
    const int4 head = st->head[e];
    f[k] = head.x;
    o[k] = in_range(xrow[head.x], head.y, (unsigned)head.z);
    if constexpr (sizeof(T) == 4) z[k] = __int_as_float(head.w);
    else z[k] = st->aux[e].z;
    w[k] = st->w(e);
    on[k] = real;
  }
}

// E_k = coefficients of prod_{k<Q} (z_k + o_k t)
template <typename T, int Q>
__device__ __forceinline__ void extend_all(const bool (&o)[Q], const T (&z)[Q], T (&E)[Q + 1]) {
  E[0] = T(1);
#pragma unroll
  for (int k = 1; k <= Q; ++k) E[k] = T(0);
#pragma unroll
  for (int l = 1; l <= Q; ++l) {
    const T zl = z[l - 1];
    const bool ol = o[l - 1];
    E[l] = ol ? E[l - 1] : T(0);
#pragma unroll
    for (int k = l - 1; k >= 1; --k) E[k] = fma(zl, E[k], ol ? E[k - 1] : T(0));
    E[0] = zl * E[0];
  }
}

// D = E / (zi + t) for a degree-Q polynomial E; D has Q terms.
template <typename T, int Q>
__device__ __forceinline__ void unwind_one(const T (&E)[Q + 1], T zi, T (&D)[Q]) {
  D[Q - 1] = E[Q];
#pragma unroll
  for (int k = Q - 1; k >= 1; --k) D[k - 1] = fma(-zi, D[k], E[k]);
}

// ---------------------------------------------------------------------------
// per-lane path arithmetic
// ---------------------------------------------------------------------------

// SHAP values.  With D^i = E / (z_i + t) (synthetic division from the top,
// D^i_k = sum_{j>k} E_j (-z_i)^{j-1-k}), the unwound sum of element i is
// sum_k c_k D^i_k = sum_m (-z_i)^m G_m with G_m = sum_{j>m} c_{j-1-m} E_j.
// phi[f_i] += v (1 - z_i) * that sum when o_i = 1, and -v sum_k c_k E_k
// when o_i = 0.
// C: the arithmetic's type (T, or double for paths of 13-16 features).
template <typename T, int Q, AddMode MODE, typename C = T>
__device__ __forceinline__ void shap_math(const int (&f)[Q], const bool (&o)[Q], const T (&z)[Q],
                                          const T (&w)[Q], const bool (&on)[Q], T v,
                                          T* __restrict__ prow) {
  C zc[Q];
#pragma unroll
  for (int k = 0; k < Q; ++k) zc[k] = C(z[k]);
  C E[Q + 1];
  extend_all<C, Q>(o, zc, E);
  C t_all = C(0);
#pragma unroll
  for (int k = 0; k < Q; ++k) t_all = fma(C(shapley_weight(Q, k)), E[k], t_all);
  C G[Q];
#pragma unroll
  for (int m = 0; m < Q; ++m) {
    G[m] = C(shapley_weight(Q, Q - 1 - m)) * E[Q];
#pragma unroll
    for (int j = Q - 1; j > m; --j) G[m] = fma(C(shapley_weight(Q, j - 1 - m)), E[j], G[m]);
  }
  const C neg_vt = -C(v) * t_all;
  T* p[Q];
  T val[Q];
#pragma unroll
  for (int i = 0; i < Q; ++i) {
    C s = G[Q - 1];
#pragma unroll
    for (int m = Q - 2; m >= 0; --m) s = fma(-zc[i], s, G[m]);
    C a = C(w[i]) * s;
    // several paths per wave: the lanes rarely agree on o_i, so a branch
    // around the Horner evaluation only adds its cost (one path per wave:
    // whole waves often have o_i = 0 and skip it)
    if constexpr (MODE == kPaired) keep(a);
    val[i] = T(o[i] ? a : neg_vt);
    p[i] = prow + f[i];
  }
  tile_add<MODE>(p, val, on);
}

// Interaction values.  For elements i != c the interaction through this path
// is Delta_ic = v/2 (o_i - z_i)(o_c - z_c) S_ic, S_ic the Shapley-weighted sum
// over the path without i and c (weights for q-1 players).  By cases on
// (o_i, o_c):
//   (1,1): S_ic from E / ((z_i + t)(z_c + t))
//   (1,0): (o_c - z_c) S_ic = -sum_k c'_k D^i_k         (D^i = E / (z_i + t))
//   (0,0): (o_i - z_i)(o_c - z_c) S_ic = sum_k c'_k E_k
// and phi_ii = phi_i - sum_{c != i} Delta_ic (Eq. 6).  Each pair is added to
// the entry [f_i][f_c] only; the tile write adds the mirror entries.  The
// lone-element values and v/2 (1 - z) are formed once per element, not once
// per pair.
template <typename T, int Q, AddMode MODE>
__device__ __forceinline__ void inter_math(const int (&f)[Q], const bool (&o)[Q], const T (&z)[Q],
                                           const T (&w)[Q], const bool (&on)[Q], T v,
                                           T* __restrict__ prow, int stride) {
  T E[Q + 1];
  extend_all<T, Q>(o, z, E);
  T t_all = T(0);
#pragma unroll
  for (int k = 0; k < Q; ++k) t_all = fma(T(shapley_weight(Q, k)), E[k], t_all);
  T t_pair = T(0);
  if constexpr (Q >= 2) {
#pragma unroll
    for (int k = 0; k < Q - 1; ++k) t_pair = fma(T(shapley_weight(Q - 1, k)), E[k], t_pair);
  }
  const T half_v = T(0.5) * v;
  const T k00 = half_v * t_pair;   // (o_i, o_c) = (0, 0)
  T lone[Q];  // -v (1 - z_c) tp[c] / 2: the pair value when only c is present
  T diag[Q];  // running phi_cc
#pragma unroll
  for (int c = 0; c < Q; ++c) {
    T D[Q];
    unwind_one<T, Q>(E, z[c], D);
    T s = T(0);
#pragma unroll
    for (int k = 0; k < Q; ++k) s = fma(T(shapley_weight(Q, k)), D[k], s);
    diag[c] = o[c] ? w[c] * s : -v * t_all;
    T tpc = T(0);
    if constexpr (Q >= 2) {
#pragma unroll
      for (int k = 0; k < Q - 1; ++k) tpc = fma(T(shapley_weight(Q - 1, k)), D[k], tpc);
    }
    const T cw = T(0.5) * w[c];   // v (1 - z_c) / 2, times (1 - z_i) below
    lone[c] = -cw * tpc;
    if (c == 0) continue;
    // S_ic for every i < c: the Shapley-weighted sum (q-1 players) of
    // D / (z_i + t).  For many i, as a polynomial in -z_i with coefficients
    // H_m = sum_k c'_k D_{k+m+1}; for few, by synthetic division.
    constexpr int kHorner = Q / 2 + 1;
    T H[Q];
    if (c > kHorner) {
#pragma unroll
      for (int m = 0; m + 1 < Q; ++m) {
        H[m] = T(shapley_weight(Q - 1, 0)) * D[m + 1];
#pragma unroll
        for (int k = 1; k + m + 1 < Q; ++k) H[m] = fma(T(shapley_weight(Q - 1, k)), D[k + m + 1], H[m]);
      }
    }
    T* p[Q];
    T val[Q];
    bool pon[Q];
#pragma unroll
    for (int i = 0; i < Q; ++i) {
      p[i] = prow;
      val[i] = T(0);
      pon[i] = false;
    }
#pragma unroll
    for (int i = 0; i < c; ++i) {
      T s11 = T(0);
      if constexpr (Q >= 2) {
        if (c > kHorner) {
          s11 = H[Q - 2];
#pragma unroll
          for (int m = Q - 3; m >= 0; --m) s11 = fma(-z[i], s11, H[m]);
        } else {
          T DD[Q];
          DD[Q - 2] = D[Q - 1];
#pragma unroll
          for (int k = Q - 2; k >= 1; --k) DD[k - 1] = fma(-z[i], DD[k], D[k]);
#pragma unroll
          for (int k = 0; k < Q - 1; ++k) s11 = fma(T(shapley_weight(Q - 1, k)), DD[k], s11);
        }
      }
      const T both = (cw * (T(1) - z[i])) * s11;
      const T delta = o[i] ? (o[c] ? both : lone[i]) : (o[c] ? lone[c] : k00);
      diag[c] -= delta;
      diag[i] -= delta;
      pon[i] = on[i] && on[c];
      p[i] = prow + tri_at(f[i], f[c], stride);
      val[i] = delta;
    }
    tile_add<MODE == kExclusive ? kExclusive : kBatched>(p, val, pon);
  }
  T* p[Q];
#pragma unroll
  for (int c = 0; c < Q; ++c) p[c] = prow + tri_row(f[c], stride) + f[c];
  tile_add<MODE>(p, diag, on);
}

// Paths longer than the unrolled variants: the same arithmetic with runtime
// loops, always in fp64, unwinding by explicit synthetic division.  Dividing
// the weight polynomial from its top coefficient down cancels more and more
// as paths grow; in fp32 the error passes the parity bound beyond about 16
// features, in fp64 it stays far inside it for the longest path a wave64
// holds (63 features).  FP64 FMAs run at the rate of unpacked FP32 ones on
// gfx950.  q = 0 (no path) does nothing.
template <typename T, bool INTER, AddMode MODE, bool GAPPED>
__device__ void path_dyn(const Stage<T, GAPPED>* st, int s, int q, const int* __restrict__ xrow,
                         T* __restrict__ prow, int stride) {
  double E[kMaxPathLen];
  double z[kMaxPathLen];
  double D[kMaxPathLen];
  int f[kMaxPathLen];
  uint64_t obits = 0;
  for (int k = 0; k < q; ++k) {
    const int4 head = st->head[s + 1 + k];
    f[k] = head.x;
    z[k] = (double)st->z(s + 1 + k);
    obits |= (uint64_t)in_range(xrow[head.x], head.y, (unsigned)head.z) << k;
  }
  const double v = (double)st->w(s);
  E[0] = 1.0;
  for (int l = 1; l <= q; ++l) {
    const double zl = z[l - 1];
    const bool ol = (obits >> (l - 1)) & 1u;
    E[l] = ol ? E[l - 1] : 0.0;
    for (int k = l - 1; k >= 1; --k) E[k] = fma(zl, E[k], ol ? E[k - 1] : 0.0);
    E[0] = zl * E[0];
  }
  double t_all = 0.0;
  for (int k = 0; k < q; ++k) t_all = fma(shapley_weight(q, k), E[k], t_all);
  if constexpr (!INTER) {
    for (int i = 0; i < q; ++i) {
      D[q - 1] = E[q];
      for (int k = q - 1; k >= 1; --k) D[k - 1] = fma(-z[i], D[k], E[k]);
      double s = 0.0;
      for (int k = 0; k < q; ++k) s = fma(shapley_weight(q, k), D[k], s);
      const bool oi = (obits >> i) & 1u;
      const double phi = oi ? v * (1.0 - z[i]) * s : -v * t_all;
      acc_add<MODE == kExclusive>(&prow[f[i]], (T)phi);
    }
  } else {
    double DD[kMaxPathLen];
    double tp[kMaxPathLen];
    double diag[kMaxPathLen];
    double t_pair = 0.0;
    for (int k = 0; k < q - 1; ++k) t_pair = fma(shapley_weight(q - 1, k), E[k], t_pair);
    const double half_v = 0.5 * v;
    for (int c = 0; c < q; ++c) {
      D[q - 1] = E[q];
      for (int k = q - 1; k >= 1; --k) D[k - 1] = fma(-z[c], D[k], E[k]);
      double s = 0.0, acc = 0.0;
      for (int k = 0; k < q; ++k) s = fma(shapley_weight(q, k), D[k], s);
      for (int k = 0; k < q - 1; ++k) acc = fma(shapley_weight(q - 1, k), D[k], acc);
      const bool oc = (obits >> c) & 1u;
      diag[c] = oc ? v * (1.0 - z[c]) * s : -v * t_all;
      tp[c] = acc;
      for (int i = 0; i < c; ++i) {
        DD[q - 2] = D[q - 1];
        for (int k = q - 2; k >= 1; --k) DD[k - 1] = fma(-z[i], DD[k], D[k]);
        double s11 = 0.0;
        for (int k = 0; k < q - 1; ++k) s11 = fma(shapley_weight(q - 1, k), DD[k], s11);
        const bool oi = (obits >> i) & 1u;
        double delta;
        if (oi && oc) delta = half_v * (1.0 - z[i]) * (1.0 - z[c]) * s11;
        else if (oi) delta = -half_v * (1.0 - z[i]) * tp[i];
        else if (oc) delta = -half_v * (1.0 - z[c]) * tp[c];
        else delta = half_v * t_pair;
        diag[c] -= delta;
        diag[i] -= delta;
        acc_add<MODE == kExclusive>(&prow[tri_at(f[i], f[c], stride)], (T)delta);
      }
    }
    for (int c = 0; c < q; ++c)
      acc_add<MODE == kExclusive>(&prow[tri_row(f[c], stride) + f[c]], (T)diag[c]);
  }
}

template <typename T, int Q, bool UNIFORM, bool INTER, AddMode MODE, bool GAPPED, typename C = T>
__device__ __forceinline__ void path_fixed(const Stage<T, GAPPED>* st, int s, int q,
                                           const int* __restrict__ xrow, T* __restrict__ prow,
                                           int stride) {
  int f[Q];
  bool o[Q], on[Q];
  T z[Q], w[Q];
  load_path<T, Q, UNIFORM, GAPPED>(st, s, q, xrow, f, o, z, w, on);
  const T v = st->w(s);
  if constexpr (INTER) inter_math<T, Q, MODE>(f, o, z, w, on, v, prow, stride);
  else shap_math<T, Q, MODE, C>(f, o, z, w, on, v, prow);
}

// Q = features of the longest path in the wave's current set (uniform); q =
// this lane's path (0: none).  QMAX = the kernel variant's longest path: the
// runtime-length code exists only in the kQLong variants.
template <typename T, bool UNIFORM, bool INTER, AddMode MODE, bool GAPPED, int QMAX>
__device__ __forceinline__ void dispatch(int Q, const Stage<T, GAPPED>* st, int s, int q,
                                         const int* xrow, T* prow, int stride) {
  static_assert(kMaxUnrolledShap == 12 && kMaxUnrolledShapF64 == 16 && kMaxUnrolledInter == 8,
                "update the case lists");
  static_assert(QMAX == kQShort || QMAX == kQMid || QMAX == kQExt || QMAX == kQLong,
                "unknown variant");
#define GTS_CASE(n) \
  case n: path_fixed<T, n, UNIFORM, INTER, MODE, GAPPED>(st, s, q, xrow, prow, stride); break;
#define GTS_CASE64(n) \
  case n: path_fixed<T, n, UNIFORM, false, MODE, GAPPED, double>(st, s, q, xrow, prow, stride); break;
  switch (Q) {
    GTS_CASE(1) GTS_CASE(2) GTS_CASE(3) GTS_CASE(4) GTS_CASE(5) GTS_CASE(6)
    GTS_CASE(7) GTS_CASE(8)
    default:
      if constexpr (!INTER && QMAX >= kQMid) {
        switch (Q) {
          GTS_CASE(9) GTS_CASE(10) GTS_CASE(11) GTS_CASE(12)
          default:
            if constexpr (QMAX >= kQExt) {
              switch (Q) {
                GTS_CASE64(13) GTS_CASE64(14) GTS_CASE64(15) GTS_CASE64(16)
                default:
                  if constexpr (QMAX == kQLong)
                    path_dyn<T, false, MODE, GAPPED>(st, s, q, xrow, prow, stride);
                  break;
              }
            }
            break;
        }
      } else if constexpr (QMAX == kQLong) {
        path_dyn<T, INTER, MODE, GAPPED>(st, s, q, xrow, prow, stride);
      }
      break;
  }
#undef GTS_CASE
#undef GTS_CASE64
}

// Largest value of v over the wave (v in [0, 64)), from six ballots.
__device__ __forceinline__ int wave_max_small(int v) {
  int m = 0;
#pragma unroll
  for (int bit = 5; bit >= 0; --bit) {
    const int c = m | (1 << bit);
    if (__ballot(v >= c)) m = c;
  }
  return m;
}

// Whether any lane's row lies inside all n0 zero-fraction elements of the
// path whose root is lane rl of the bin (its elements rl+1 .. rl+n0, held by
// those lanes of b; the bin is a wave-uniform unit).  A row outside one of
// them meets a factor z + o t = 0: every weight of that (row, path) is 0, and
// so is its every contribution.  The elements' fields come from their lanes'
// registers; two elements are tested per LDS round trip for the rows' x.
template <typename T>
__device__ __forceinline__ bool wave_live(const Bin<T>& b, int rl, int n0,
                                          const int* __restrict__ xrow) {
  // two elements per step (the last one twice when n0 is odd).  A row's miss
  // is all ones once it fails a test; folded into the key distance of the
  // next test, it fails that one too, so one compare per step decides.
  unsigned miss = 0u;
  for (int k = 0; k < n0; k += 2) {
    const int e1 = rl + 1 + k;
    const int e2 = rl + 1 + min(k + 1, n0 - 1);
    const int f1 = __builtin_amdgcn_readlane(b.feat, e1);
    const int f2 = __builtin_amdgcn_readlane(b.feat, e2);
    const int klo1 = __builtin_amdgcn_readlane(b.klo, e1);
    const int klo2 = __builtin_amdgcn_readlane(b.klo, e2);
    const unsigned span1 = (unsigned)__builtin_amdgcn_readlane((int)b.span, e1);
    const unsigned span2 = (unsigned)__builtin_amdgcn_readlane((int)b.span, e2);
    const unsigned d1 = (unsigned)xrow[f1] - (unsigned)klo1;
    const unsigned d2 = (unsigned)xrow[f2] - (unsigned)klo2;
    miss |= d1 < span1 ? 0u : ~0u;
    const unsigned m = d2 | miss;
    // lanes still inside every range so far, straight from the compare
    if (__builtin_amdgcn_uicmp(m, span2, 36 /* unsigned less than */) == 0) return false;
    miss = m < span2 ? 0u : ~0u;
  }
  return true;
}

// Rank tables of a 64-row tile, per feature f < M: keys[f][p] = the p-th
// smallest row key (ties in row order) and below[f][p] = the mask of the rows
// of ranks < p (p = 0..64).  Both have rows of 65 entries, so lanes that
// probe the same rank of different features read different LDS banks (rows
// of 64 keys: 3.13 against 2.78 ms for the deep model).  The rows whose key lies in [klo, khi) are then
// below[f][c] & ~below[f][a] with a, c the numbers of keys < klo and < khi.
// Wave w builds the tables of features w, w + WAVES, ...
struct RankTables {
  uint64_t* below;   // [M][65]
  int* keys;         // [M][65], the last entry unused
  __device__ RankTables(unsigned char* base, int M)
      : below(reinterpret_cast<uint64_t*>(base)),
        keys(reinterpret_cast<int*>(base + (size_t)M * 65 * sizeof(uint64_t))) {}
};

template <int WAVES>
__device__ void build_ranks(const int* xs, int sx, int M, RankTables rt, int wave, int lane) {
  for (int f = wave; f < M; f += WAVES) {
    const int kx = xs[lane * sx + f];
    int rank = 0;
#pragma unroll 16
    for (int j = 0; j < 64; ++j) {
      const int kj = __builtin_amdgcn_readlane(kx, j);
      rank += (kj < kx || (kj == kx && j < lane)) ? 1 : 0;
    }
    rt.keys[f * 65 + rank] = kx;
    // lane p takes the row of rank p; the masks are an inclusive OR-scan of
    // the rows' bits in rank order
    const int row = __builtin_amdgcn_ds_permute(rank * 4, lane);
    unsigned lo = row < 32 ? 1u << row : 0u;
    unsigned hi = row >= 32 ? 1u << (row - 32) : 0u;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const unsigned ulo = __shfl_up(lo, d);
      const unsigned uhi = __shfl_up(hi, d);
      if (lane >= d) {
        lo |= ulo;
        hi |= uhi;
      }
    }
    rt.below[f * 65 + lane + 1] = (uint64_t)hi << 32 | lo;
    if (lane == 0) rt.below[f * 65] = 0;
  }
}

// Roots of the bin's paths that some row of the tile reaches: every lane
// holding a zero-fraction element finds the rows inside its range from the
// rank tables (two binary searches), and each root lane intersects the row
// sets of its path's zero-fraction elements (stored right after it).  The
// same test as wave_live, for all paths of the bin at once.
template <typename T, int QMAX>
__device__ __forceinline__ uint64_t live_roots(const Bin<T>& b, int lane, uint64_t roots,
                                               int info, RankTables rt) {
  uint64_t rows = ~0ull;
  if (lane < b.len && b.feat >= 0 && b.z == T(0)) {
    const int* ks = rt.keys + b.feat * 65;
    const int klo = b.klo;
    const int khi = (int)((unsigned)b.klo + b.span);
    int a = 0, c = 0;
#pragma unroll
    for (int s = 32; s >= 1; s >>= 1) {
      a += ks[a + s - 1] < klo ? s : 0;
      c += ks[c + s - 1] < khi ? s : 0;
    }
    a += ks[a] < klo ? 1 : 0;
    c += ks[c] < khi ? 1 : 0;
    rows = rt.below[b.feat * 65 + c] & ~rt.below[b.feat * 65 + a];
  }
  // AND over each path's lanes (its root and its non-zero-fraction
  // elements hold all ones): a segmented suffix scan, steps of 1, 2, 4, ...
  // lanes while no root lies in between; four steps cover paths of up to 16
  // elements, five up to 32
  unsigned lo = (unsigned)rows, hi = (unsigned)(rows >> 32);
  const uint64_t later = lane < 63 ? roots >> (lane + 1) : 0ull;   // roots above this lane
  constexpr int kSteps = QMAX <= kQMid ? 4 : QMAX <= kQExt ? 5 : 6;
#pragma unroll
  for (int t = 0; t < kSteps; ++t) {
    const int d = 1 << t;
    const unsigned nlo = __shfl_down(lo, d);
    const unsigned nhi = __shfl_down(hi, d);
    if ((later & ((1ull << d) - 1ull)) == 0) {
      lo &= nlo;
      hi &= nhi;
    }
  }
  const bool root = (roots >> lane) & 1ull;
  return __ballot(root && (info & 0xff) > 0 && (lo | hi) != 0u);
}

// All paths of one bin.  RW == 64: one path at a time for the whole wave,
// skipped when no row of the tile reaches its zero-fraction ranges.  RW < 64:
// rounds of up to P = 64/RW paths, lane (j, r) = (path j, row r).  (Finding
// the dead paths of a bin first and leaving them out of the rounds was
// measured slower: a round is saved only when the live paths fit in fewer
// rounds, and the test of every path costs more than that saves.)
template <typename T, int RW, bool INTER, bool EXCL, int QMAX>
__device__ __forceinline__ void process_bin(Stage<T, RW < 64>* st, const Bin<T>& b, int lane,
                                            const int* xrow, T* prow, int stride, bool sorted,
                                            bool ranked, RankTables rt) {
  const BinIndex ix = index_bin(b, lane);
  const uint64_t roots = ix.roots;
  const int info = ix.info;
  if constexpr (RW == 64) {
    // paths from the roots' ballot, each word from its root lane; in the
    // ungapped stage, slot = lane.  With rank tables the live paths are
    // known for the whole bin at once, before staging: a bin with none is
    // not staged at all.
    uint64_t rest = roots;
    if (ranked) {
      rest = live_roots<T, QMAX>(b, lane, roots, info, rt);
      if (rest == 0) return;
    }
    stage_bin(st, b, lane, ix);
    while (rest != 0) {
      const int rl = __builtin_ctzll(rest);
      rest &= rest - 1ull;
      const int word = __builtin_amdgcn_readlane(info, rl);
      const int q = word & 0xff;
      const int n0 = word >> 8;
      if (ranked || (q > 0 && (n0 == 0 || wave_live(b, rl, n0, xrow))))
        dispatch<T, true, INTER, EXCL ? kExclusive : kBatched, false, QMAX>(q, st, rl, q, xrow,
                                                                             prow, stride);
    }
  } else {
    constexpr int P = 64 / RW;
    const int j = lane / RW;
    const int npaths = stage_bin(st, b, lane, ix);
    for (int base = 0; base < npaths; base += P) {
      const int t = base + j;
      const bool valid = t < npaths;
      const int info = valid ? st->path[t] : 0;
      const int my_s = path_slot(info);
      const int my_q = path_q(info);
      // the round's longest path: its first when the bin's paths never grow
      const int qmax = sorted ? path_q(__builtin_amdgcn_readfirstlane(st->path[base]))
                              : wave_max_small(my_q);
      if (qmax > 0)
        dispatch<T, false, INTER, kPaired, true, QMAX>(qmax, st, my_s, my_q, xrow, prow, stride);
    }
  }
  // the next bin overwrites the stage
  __builtin_amdgcn_wave_barrier();
}

// One workgroup: rows [tile*RW, tile*RW + RW) of output group g, bins of
// slice s of that group (every splits-th bin, starting at bin s).  PRIV:
// every wave accumulates into a phi tile of its own (summed when the tile is
// written), so waves never contend; with one path per wave (RW == 64) the
// accumulation then needs no atomics.  Workgroups are dealt to the 8 XCDs
// round-robin.  When the (group, slice) units divide evenly among the XCDs,
// consecutive workgroups on an XCD take the same unit for successive row
// tiles; otherwise the grid is unit-major, all XCDs working through one
// unit's row tiles together.  Either way each XCD's L2 holds about one
// unit's bins at a time.
template <typename T, int RW, bool INTER, int WAVES, bool PRIV, int QMAX>
__global__ __launch_bounds__(64 * WAVES) void shap_kernel(DevModel<T> d, const float* __restrict__ X,
                                                         T* __restrict__ phi, Launch L) {
  extern __shared__ __align__(16) unsigned char smem[];
  constexpr int kThreads = 64 * WAVES;
  const int M = d.M;
  const int G = d.G;
  const int U = G * L.splits;
  const int64_t b = blockIdx.x;
  int64_t tile;
  int u;
  if (U % 8 == 0) {
    const int64_t local = b >> 3;
    tile = local % L.tiles;
    u = (int)(b & 7) + 8 * (int)(local / L.tiles);
  } else {
    // unit-major: the XCDs work through one unit's row tiles together, so
    // each L2 holds the bins of about one unit at a time
    tile = b % L.tiles;
    u = (int)(b / L.tiles);
  }
  const int g = u / L.splits;
  const int s = u - g * L.splits;
  const int64_t r0 = tile * RW;
  const int gb0 = d.group_bins[g];
  const int gb1 = d.group_bins[g + 1];
  int b_step = L.splits;
  if (L.adaptive) {
    // each wave about 32 bins or more; at least the occupancy target
    const int fine = (gb1 - gb0) / (32 * WAVES) / L.split_step * L.split_step;
    b_step = min(L.splits, max(L.min_splits, fine));
    if (s >= b_step) return;   // the whole workgroup, before any barrier
  }

  int* xs = reinterpret_cast<int*>(smem);   // the X tile, as fkey of each value
  T* ps = reinterpret_cast<T*>(smem + (size_t)RW * L.sx * sizeof(float));
  constexpr int NT = PRIV ? WAVES : 1;  // phi tiles
  const int tile_elems = RW * L.sp;
  Stage<T, RW < 64>* stages = reinterpret_cast<Stage<T, RW < 64>*>(
      smem + (((size_t)RW * L.sx * sizeof(float) + (size_t)NT * tile_elems * sizeof(T) + 15) & ~(size_t)15));

  // stage the X tile (coalesced along each row) and clear the phi tile
  for (int i = threadIdx.x; i < RW * M; i += kThreads) {
    const int r = i / M, c = i - r * M;
    const int64_t row = r0 + r;
    xs[r * L.sx + c] = fkey(row < L.rows ? X[row * L.ld + c] : 0.0f);
  }
  for (int i = threadIdx.x; i < NT * tile_elems; i += kThreads) ps[i] = T(0);
  __syncthreads();

  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  // rank tables: only the private-tile launches (one path per wave, small
  // M) have them, so the other variants carry none of their code
  const bool ranked = PRIV && RW == 64 && L.rank_off > 0;
  const RankTables rt(smem + L.rank_off, M);
  if (ranked) {
    build_ranks<WAVES>(xs, L.sx, M, rt, wave, lane);
    __syncthreads();
  }
  const int r = lane % RW;
  init_stage(stages + wave, lane);
  // Slice s takes every splits-th bin of the group.  Bins come longest paths
  // first, so contiguous runs would give the first slices the most work;
  // strided, every slice gets bins of every size.
  const int b_lo = gb0 + s;
  const int* xrow = xs + r * L.sx;
  T* prow = ps + (PRIV ? wave * tile_elems : 0) + r * L.sp;
  const int stride = M + 1;

  int bi = b_lo + wave * b_step;
  if (bi < gb1) {
    Bin<T> cur = load_bin(d, bi, lane);
    for (; bi < gb1; bi += WAVES * b_step) {
      Bin<T> nxt;
      const int bn = bi + WAVES * b_step;
      if (bn < gb1) nxt = load_bin(d, bn, lane);
      process_bin<T, RW, INTER, PRIV && RW == 64, QMAX>(stages + wave, cur, lane, xrow, prow,
                                                        stride, L.sorted != 0, ranked, rt);
      cur = nxt;
    }
  }
  __syncthreads();

  // write the tile: phi[row][g][.]; the bias goes to the last entry.  An
  // interaction entry (a, b) and its mirror (b, a) both get the triangle's
  // entry, so the output is exactly symmetric.
  const T bias = d.bias[g];
  const int W = L.width;
  for (int i = threadIdx.x; i < RW * W; i += kThreads) {
    const int rr = i / W, c = i - rr * W;
    const int64_t row = r0 + rr;
    if (row >= L.rows) continue;
    int t = c;
    if constexpr (INTER) {
      const int a = c / stride;
      t = tri_at(a, c - a * stride, stride);
    }
    T val = ps[rr * L.sp + t];
#pragma unroll
    for (int w = 1; w < NT; ++w) val += ps[w * tile_elems + rr * L.sp + t];
    if (c == W - 1 && s == 0) val += bias;
    T* out = phi + (row * G + g) * (int64_t)W + c;
    if (L.accumulate) unsafeAtomicAdd(out, val);
    else *out = val;
  }
}

template <typename T>
__global__ void fill_zero(T* __restrict__ p, int64_t n) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) p[i] = T(0);
}


// ---------------------------------------------------------------------------
// launch of one variant
// ---------------------------------------------------------------------------

template <typename T, int RW, bool INTER, int WAVES, bool PRIV, int QMAX>
gts_status launch_rw(const KernelArgs& a, const Plan& p) {
  const gts_model* m = a.m;
  hipStream_t stream = static_cast<hipStream_t>(a.stream);
  DevModel<T> d = dev_model<T>(m, a.blob);
  Launch L;
  L.rows = a.rows;
  L.ld = a.ld;
  L.tiles = (int32_t)((a.rows + RW - 1) / RW);
  L.splits = p.splits;
  L.sx = p.sx;
  L.sp = p.sp;
  L.width = p.width;
  L.accumulate = p.splits > 1 ? 1 : 0;
  L.sorted = (m->flags & GTS_MODEL_SORTED_BINS) ? 1 : 0;
  L.rank_off = (int32_t)p.rank_off;
  L.adaptive = (m->flags & GTS_MODEL_PRUNED) ? 1 : 0;
  L.min_splits = p.min_splits;
  L.split_step = p.split_step;
  const int64_t total = a.rows * (int64_t)m->num_groups * p.width;
  if (L.accumulate) {
    const int64_t blocks = std::min<int64_t>((total + 255) / 256, 65536);
    hipLaunchKernelGGL(fill_zero<T>, dim3((unsigned)blocks), dim3(256), 0, stream,
                       static_cast<T*>(a.phi), total);
  }
  const int64_t grid = (int64_t)L.tiles * m->num_groups * p.splits;
  if (grid > 0x7fffffffLL) return fail(GTS_EINVAL, "problem too large for one launch");
  auto kern = shap_kernel<T, RW, INTER, WAVES, PRIV, QMAX>;
  if (hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                          hipFuncAttributeMaxDynamicSharedMemorySize, (int)p.lds) != hipSuccess) {
    (void)hipGetLastError();   // leave no error behind for the caller's next HIP call
    return fail(GTS_EDEVICE, "cannot set the LDS size of the kernel to %zu bytes", p.lds);
  }
  hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(64 * WAVES), p.lds, stream, d, a.X,
                     static_cast<T*>(a.phi), L);
  const hipError_t err = hipGetLastError();
  if (err != hipSuccess) return fail(GTS_EDEVICE, "kernel launch failed: %s", hipGetErrorString(err));
  return GTS_OK;
}

template <typename T, bool INTER, int QMAX>
gts_status launch_shape(const KernelArgs& a, const Plan& p) {
  if (p.priv) return launch_rw<T, 64, INTER, 4, true, QMAX>(a, p);
#define GTS_LAUNCH(rw, w) return launch_rw<T, rw, INTER, w, false, QMAX>(a, p)
  switch (p.RW) {
    case 64: GTS_LAUNCH(64, 8);
    case 32: GTS_LAUNCH(32, 8);
    case 16:
      if (p.waves == 12) GTS_LAUNCH(16, 12);
      if (p.waves == 16) GTS_LAUNCH(16, 16);
      GTS_LAUNCH(16, 8);
    case 8:
      if (p.waves == 12) GTS_LAUNCH(8, 12);
      if (p.waves == 16) GTS_LAUNCH(8, 16);
      GTS_LAUNCH(8, 8);
    default:
      if (p.waves == 12) GTS_LAUNCH(4, 12);
      if (p.waves == 16) GTS_LAUNCH(4, 16);
      GTS_LAUNCH(4, 8);
  }
#undef GTS_LAUNCH
}

// The variant for the model's longest path.
template <typename T, bool INTER>
gts_status launch_plan(const KernelArgs& a, const Plan& p) {
  if (p.qmax <= kQShort) return launch_shape<T, INTER, kQShort>(a, p);
  if constexpr (!INTER) {
    if (p.qmax <= kQMid) return launch_shape<T, INTER, kQMid>(a, p);
    if (p.qmax <= kQExt) return launch_shape<T, INTER, kQExt>(a, p);
  }
  return launch_shape<T, INTER, kQLong>(a, p);
}

}  // namespace
}  // namespace gts
