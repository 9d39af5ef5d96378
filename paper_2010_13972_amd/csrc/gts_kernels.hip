// Device half of libgts for gfx950 (CDNA4, wave64): SHAP values and SHAP
// interaction values of merged tree paths.
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
// compile-time constants (one variant per path length up to 12 features, 8
// for interactions), so a wave never diverges on path length.  This does the
// q^2 work of a path once per row instead of spreading it over q lanes that
// then need q shuffles each.
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
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <mutex>
#include <numeric>
#include <type_traits>
#include <vector>

#include "gts_internal.h"

namespace gts {
namespace {

constexpr int kMaxUnrolledShap = 12;   // longest path (features) with unrolled code
constexpr int kMaxUnrolledInter = 8;

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
  int32_t sp;        // LDS row stride of the phi tile (elements)
  int32_t width;     // phi entries per (row, group): M+1 or (M+1)^2
  int32_t accumulate;  // 1: atomically add the tile to phi (phi pre-zeroed)
  int32_t sorted;      // 1: inside a bin, paths never grow in length
};

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
#pragma unroll
      for (int i = 0; i < N; ++i) {
        old[i] = *reinterpret_cast<const U*>(p[i]);
        got[i] = on[i] ? atomicCAS(reinterpret_cast<U*>(p[i]), old[i],
                                   Bits<T>::of(Bits<T>::val(old[i]) + val[i]))
                       : old[i];
      }
    }
    bool retry = false;
#pragma unroll
    for (int i = 0; i < N; ++i) retry |= got[i] != old[i];
    if (retry) {
#pragma unroll
      for (int i = 0; i < N; ++i)
        if (got[i] != old[i]) lds_add(p[i], val[i]);
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
  int feat;   // -1 root, -2 past the end of the bin
  float lo, hi;
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
    b.lo = d.lower[e];
    b.hi = d.upper[e];
    b.z = d.zero[e];
  } else {
    b.feat = -2;
    b.lo = 0.0f;
    b.hi = 0.0f;
    b.z = T(0);
  }
  return b;
}

// One wave's copy of its current bin in LDS.  head[slot] = (feature, lower
// bits, upper bits, fp32 z bits); aux[slot] holds w = v (1 - z), v the leaf
// value of the element's path (and z itself for fp64 models); on a root, z
// and w hold v.  path[t] = slot of the t-th root | (features of its path) << 8.
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
    st->head[S::kSlots] = make_int4(0, __float_as_int(-INFINITY), __float_as_int(INFINITY),
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

template <typename T, bool GAPPED>
__device__ __forceinline__ int stage_bin(Stage<T, GAPPED>* st, const Bin<T>& b, int lane) {
  const bool root = b.feat == -1;
  const uint64_t roots = __ballot(root);
  const uint64_t upto = roots & ((2ull << lane) - 1ull);      // roots at or below this lane
  const int rl = upto ? 63 - __clzll((long long)upto) : lane;  // this element's root
  const uint64_t above = roots & ~((2ull << lane) - 1ull);
  const int len = (above ? __builtin_ctzll(above) : b.len) - lane;  // path length, on a root
  int slot = lane;
  if constexpr (GAPPED) {
    const uint64_t evens = __ballot(root && (len & 1) == 0);
    slot += __popcll(evens & ((1ull << rl) - 1ull));
  }
  const T v = __shfl(b.z, rl);   // a root's zero-fraction slot holds v
  const T w = root ? v : v * (T(1) - b.z);
  st->head[slot] = make_int4(b.feat, __float_as_int(b.lo), __float_as_int(b.hi),
                             sizeof(T) == 4 ? __float_as_int((float)b.z) : 0);
  typename Stage<T, GAPPED>::AuxT ax{};
  if constexpr (std::is_same_v<typename Stage<T, GAPPED>::AuxT, float>) {
    ax = w;
  } else {
    if constexpr (sizeof(T) == 8) ax.z = b.z;
    ax.w = w;
  }
  st->aux[slot] = ax;
  const int rank = __builtin_amdgcn_mbcnt_hi((unsigned)(roots >> 32),
                                             __builtin_amdgcn_mbcnt_lo((unsigned)roots, 0u));
  if (root) st->path[rank] = slot | ((len - 1) << 8);
  // the stores above are read by other lanes of this wave only
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  return __popcll(roots);
}

// Feature, presence test o_k = [lower <= x < upper], zero fraction and
// v (1 - z) of the first Q feature elements of the path whose root is in
// slot s (wave-uniform when UNIFORM).  A lane whose path has q < Q features
// reads the neutral element for k >= q; on[k] = k < q marks the elements
// whose contributions are written.
template <typename T, int Q, bool UNIFORM, bool GAPPED>
__device__ __forceinline__ void load_path(const Stage<T, GAPPED>* st, int s, int q,
                                          const float* __restrict__ xrow, int (&f)[Q],
                                          bool (&o)[Q], T (&z)[Q], T (&w)[Q], bool (&on)[Q]) {
#pragma unroll
  for (int k = 0; k < Q; ++k) {
    const bool real = UNIFORM || k < q;
    const int e = real ? s + 1 + k : Stage<T, GAPPED>::kSlots;
    const int4 head = st->head[e];
    f[k] = head.x;
    const float x = xrow[head.x];
    o[k] = (__int_as_float(head.y) <= x) && (x < __int_as_float(head.z));
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
template <typename T, int Q, AddMode MODE>
__device__ __forceinline__ void shap_math(const int (&f)[Q], const bool (&o)[Q], const T (&z)[Q],
                                          const T (&w)[Q], const bool (&on)[Q], T v,
                                          T* __restrict__ prow) {
  T E[Q + 1];
  extend_all<T, Q>(o, z, E);
  T t_all = T(0);
#pragma unroll
  for (int k = 0; k < Q; ++k) t_all = fma(T(shapley_weight(Q, k)), E[k], t_all);
  T G[Q];
#pragma unroll
  for (int m = 0; m < Q; ++m) {
    G[m] = T(shapley_weight(Q, Q - 1 - m)) * E[Q];
#pragma unroll
    for (int j = Q - 1; j > m; --j) G[m] = fma(T(shapley_weight(Q, j - 1 - m)), E[j], G[m]);
  }
  const T neg_vt = -v * t_all;
  T* p[Q];
  T val[Q];
#pragma unroll
  for (int i = 0; i < Q; ++i) {
    T s = G[Q - 1];
#pragma unroll
    for (int m = Q - 2; m >= 0; --m) s = fma(-z[i], s, G[m]);
    val[i] = o[i] ? w[i] * s : neg_vt;
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
  T hw[Q];    // v (1 - z_i) / 2
  T zc1[Q];   // 1 - z_c
  T lone[Q];  // -v (1 - z_c) tp[c] / 2: the pair value when only c is present
  T diag[Q];  // running phi_cc
#pragma unroll
  for (int i = 0; i < Q; ++i) {
    hw[i] = T(0.5) * w[i];
    zc1[i] = T(1) - z[i];
  }
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
    lone[c] = -hw[c] * tpc;
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
    const T cw = hw[c];   // v (1 - z_c) / 2, times (1 - z_i) below
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
      const T both = (cw * zc1[i]) * s11;
      const T delta = o[i] ? (o[c] ? both : lone[i]) : (o[c] ? lone[c] : k00);
      diag[c] -= delta;
      diag[i] -= delta;
      pon[i] = on[i] && on[c];
      p[i] = prow + f[i] * stride + f[c];
      val[i] = delta;
    }
    tile_add<MODE == kExclusive ? kExclusive : kBatched>(p, val, pon);
  }
  T* p[Q];
#pragma unroll
  for (int c = 0; c < Q; ++c) p[c] = prow + f[c] * stride + f[c];
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
__device__ void path_dyn(const Stage<T, GAPPED>* st, int s, int q, const float* __restrict__ xrow,
                         T* __restrict__ prow, int stride) {
  double E[kMaxPathLen];
  double z[kMaxPathLen];
  double D[kMaxPathLen];
  int f[kMaxPathLen];
  uint64_t obits = 0;
  for (int k = 0; k < q; ++k) {
    const int4 head = st->head[s + 1 + k];
    const float x = xrow[head.x];
    f[k] = head.x;
    z[k] = (double)st->z(s + 1 + k);
    obits |= (uint64_t)((__int_as_float(head.y) <= x) && (x < __int_as_float(head.z))) << k;
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
        acc_add<MODE == kExclusive>(&prow[f[i] * stride + f[c]], (T)delta);
      }
    }
    for (int c = 0; c < q; ++c) acc_add<MODE == kExclusive>(&prow[f[c] * stride + f[c]], (T)diag[c]);
  }
}

template <typename T, int Q, bool UNIFORM, bool INTER, AddMode MODE, bool GAPPED>
__device__ __forceinline__ void path_fixed(const Stage<T, GAPPED>* st, int s, int q,
                                           const float* __restrict__ xrow, T* __restrict__ prow,
                                           int stride) {
  int f[Q];
  bool o[Q], on[Q];
  T z[Q], w[Q];
  load_path<T, Q, UNIFORM, GAPPED>(st, s, q, xrow, f, o, z, w, on);
  const T v = st->w(s);
  if constexpr (INTER) inter_math<T, Q, MODE>(f, o, z, w, on, v, prow, stride);
  else shap_math<T, Q, MODE>(f, o, z, w, on, v, prow);
}

// Q = features of the longest path in the wave's current set (uniform); q =
// this lane's path (0: none).
template <typename T, bool UNIFORM, bool INTER, AddMode MODE, bool GAPPED>
__device__ __forceinline__ void dispatch(int Q, const Stage<T, GAPPED>* st, int s, int q,
                                         const float* xrow, T* prow, int stride) {
  static_assert(kMaxUnrolledShap == 12 && kMaxUnrolledInter == 8, "update the case lists");
  if constexpr (INTER) {
    switch (Q) {
#define GTS_CASE(n) case n: path_fixed<T, n, UNIFORM, true, MODE, GAPPED>(st, s, q, xrow, prow, stride); break;
      GTS_CASE(1) GTS_CASE(2) GTS_CASE(3) GTS_CASE(4) GTS_CASE(5) GTS_CASE(6)
      GTS_CASE(7) GTS_CASE(8)
#undef GTS_CASE
      default: path_dyn<T, true, MODE, GAPPED>(st, s, q, xrow, prow, stride); break;
    }
  } else {
    switch (Q) {
#define GTS_CASE(n) case n: path_fixed<T, n, UNIFORM, false, MODE, GAPPED>(st, s, q, xrow, prow, stride); break;
      GTS_CASE(1) GTS_CASE(2) GTS_CASE(3) GTS_CASE(4) GTS_CASE(5) GTS_CASE(6)
      GTS_CASE(7) GTS_CASE(8) GTS_CASE(9) GTS_CASE(10) GTS_CASE(11) GTS_CASE(12)
#undef GTS_CASE
      default: path_dyn<T, false, MODE, GAPPED>(st, s, q, xrow, prow, stride); break;
    }
  }
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

// All paths of one bin.  RW == 64: one path at a time for the whole wave.
// RW < 64: rounds of up to P = 64/RW paths, lane (j, r) = (path j, row r).
template <typename T, int RW, bool INTER, bool EXCL>
__device__ __forceinline__ void process_bin(Stage<T, RW < 64>* st, const Bin<T>& b, int lane,
                                            const float* xrow, T* prow, int stride, bool sorted) {
  const int nroots = stage_bin(st, b, lane);
  if constexpr (RW == 64) {
    for (int t = 0; t < nroots; ++t) {
      const int info = __builtin_amdgcn_readfirstlane(st->path[t]);
      const int s = info & 0xff;
      const int q = info >> 8;
      if (q > 0) dispatch<T, true, INTER, EXCL ? kExclusive : kBatched, false>(q, st, s, q, xrow, prow, stride);
    }
  } else {
    constexpr int P = 64 / RW;
    const int j = lane / RW;
    for (int base = 0; base < nroots; base += P) {
      const int t = base + j;
      const bool valid = t < nroots;
      const int info = valid ? st->path[t] : 0;
      const int my_s = info & 0xff;
      const int my_q = info >> 8;
      // the round's longest path: its first when the bin's paths never grow
      const int qmax = sorted ? __builtin_amdgcn_readfirstlane(st->path[base]) >> 8
                              : wave_max_small(my_q);
      if (qmax > 0) dispatch<T, false, INTER, kPaired, true>(qmax, st, my_s, my_q, xrow, prow, stride);
    }
  }
  // the next bin overwrites the stage
  __builtin_amdgcn_wave_barrier();
}

// One workgroup: rows [tile*RW, tile*RW + RW) of output group g, bins of
// slice s of that group (every splits-th bin, starting at bin s).  PRIV: every wave accumulates into a phi tile of its
// own (summed when the tile is written), so waves never contend; with one
// path per wave (RW == 64) the accumulation then needs no atomics.
// Workgroups are dealt to the 8 XCDs round-robin; when the (group, slice)
// units divide evenly among the XCDs, consecutive workgroups on an XCD take
// the same unit for successive row tiles, so each XCD's L2 holds only its own
// share of the model's bins.
template <typename T, int RW, bool INTER, int WAVES, bool PRIV>
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
    tile = b / U;
    u = (int)(b % U);
  }
  const int g = u / L.splits;
  const int s = u - g * L.splits;
  const int64_t r0 = tile * RW;

  float* xs = reinterpret_cast<float*>(smem);
  T* ps = reinterpret_cast<T*>(smem + (size_t)RW * L.sx * sizeof(float));
  constexpr int NT = PRIV ? WAVES : 1;  // phi tiles
  const int tile_elems = RW * L.sp;
  Stage<T, RW < 64>* stages = reinterpret_cast<Stage<T, RW < 64>*>(
      smem + (((size_t)RW * L.sx * sizeof(float) + (size_t)NT * tile_elems * sizeof(T) + 15) & ~(size_t)15));

  // stage the X tile (coalesced along each row) and clear the phi tile
  for (int i = threadIdx.x; i < RW * M; i += kThreads) {
    const int r = i / M, c = i - r * M;
    const int64_t row = r0 + r;
    xs[r * L.sx + c] = row < L.rows ? X[row * L.ld + c] : 0.0f;
  }
  for (int i = threadIdx.x; i < NT * tile_elems; i += kThreads) ps[i] = T(0);
  __syncthreads();

  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int r = lane % RW;
  init_stage(stages + wave, lane);
  // Slice s takes every splits-th bin of the group.  Bins come longest paths
  // first, so contiguous runs would give the first slices the most work;
  // strided, every slice gets bins of every size.
  const int gb1 = d.group_bins[g + 1];
  const int b_lo = d.group_bins[g] + s;
  const int b_step = L.splits;
  const float* xrow = xs + r * L.sx;
  T* prow = ps + (PRIV ? wave * tile_elems : 0) + r * L.sp;
  const int stride = M + 1;

  int bi = b_lo + wave * b_step;
  if (bi < gb1) {
    Bin<T> cur = load_bin(d, bi, lane);
    for (; bi < gb1; bi += WAVES * b_step) {
      Bin<T> nxt;
      const int bn = bi + WAVES * b_step;
      if (bn < gb1) nxt = load_bin(d, bn, lane);
      process_bin<T, RW, INTER, PRIV && RW == 64>(stages + wave, cur, lane, xrow, prow, stride,
                                                  L.sorted != 0);
      cur = nxt;
    }
  }
  __syncthreads();

  // write the tile: phi[row][g][.]; the bias goes to the last entry.  An
  // interaction pair was added to one of its two entries: each of them gets
  // the sum of both.
  const T bias = d.bias[g];
  const int W = L.width;
  for (int i = threadIdx.x; i < RW * W; i += kThreads) {
    const int rr = i / W, c = i - rr * W;
    const int64_t row = r0 + rr;
    if (row >= L.rows) continue;
    int cm = c;
    if constexpr (INTER) {
      const int a = c / stride, bcol = c - a * stride;
      cm = bcol * stride + a;
    }
    T val = ps[rr * L.sp + c];
    if (cm != c) val += ps[rr * L.sp + cm];
#pragma unroll
    for (int w = 1; w < NT; ++w) {
      val += ps[w * tile_elems + rr * L.sp + c];
      if (cm != c) val += ps[w * tile_elems + rr * L.sp + cm];
    }
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
// host-side launch
// ---------------------------------------------------------------------------

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

template <typename T, int RW, bool INTER, int WAVES, bool PRIV>
gts_status launch_rw(const gts_model* m, const void* blob, const float* X, int64_t rows,
                     int64_t ld, void* phi, hipStream_t stream, int splits, int32_t sx, int32_t sp,
                     int32_t width, size_t lds) {
  DevModel<T> d = dev_model<T>(m, blob);
  Launch L;
  L.rows = rows;
  L.ld = ld;
  L.tiles = (int32_t)((rows + RW - 1) / RW);
  L.splits = splits;
  L.sx = sx;
  L.sp = sp;
  L.width = width;
  L.accumulate = splits > 1 ? 1 : 0;
  L.sorted = (m->flags & GTS_MODEL_SORTED_BINS) ? 1 : 0;
  const int64_t total = rows * (int64_t)m->num_groups * width;
  if (L.accumulate) {
    const int64_t blocks = std::min<int64_t>((total + 255) / 256, 65536);
    hipLaunchKernelGGL(fill_zero<T>, dim3((unsigned)blocks), dim3(256), 0, stream,
                       static_cast<T*>(phi), total);
  }
  const int64_t grid = (int64_t)L.tiles * m->num_groups * splits;
  if (grid > 0x7fffffffLL) return fail(GTS_EINVAL, "problem too large for one launch");
  auto kern = shap_kernel<T, RW, INTER, WAVES, PRIV>;
  if (hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                          hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) != hipSuccess)
    return fail(GTS_EDEVICE, "cannot set the LDS size of the kernel to %zu bytes", lds);
  hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(64 * WAVES), lds, stream, d, X,
                     static_cast<T*>(phi), L);
  const hipError_t err = hipGetLastError();
  if (err != hipSuccess) return fail(GTS_EDEVICE, "kernel launch failed: %s", hipGetErrorString(err));
  return GTS_OK;
}

// The launch shape of a model and row count: rows per tile, waves, private
// tiles, LDS strides and bytes, and bin slices.
struct Plan {
  int RW = 0;
  int waves = 8;
  bool priv = false;
  int32_t sx = 0, sp = 0, width = 0;
  size_t lds = 0;
  int splits = 1;
  int64_t tiles = 0;
};

template <typename T, bool INTER>
gts_status plan_launch(const gts_model* m, int64_t rows, const DeviceInfo& dev, Plan& plan) {
  const int M = m->num_features;
  const int G = m->num_groups;
  const int64_t width64 = INTER ? (int64_t)(M + 1) * (M + 1) : (int64_t)(M + 1);
  if (width64 > (1 << 30)) return fail(GTS_EINVAL, "M = %d is too large", M);
  const int32_t width = (int32_t)width64;
  const int32_t sx = odd_at_least(M);
  const int32_t sp = odd_at_least(width);
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
    if (RW == 0 && (int64_t)need(8, 8, false) <= dev.lds_per_block) RW = 8;
    if (RW == 0 && (int64_t)need(4, 8, false) <= dev.lds_per_block) RW = 4;
    // Waves per workgroup for a shared tile of RW <= 16 rows: as many waves
    // per CU as the LDS allows, up to 24 (the VGPR budget of the SHAP
    // kernels) or 16 (interactions).
    if (RW != 0 && RW <= 16) {
      const int cap = INTER ? 16 : 24;
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
  const size_t lds = need(RW, waves, priv);
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
  if constexpr (INTER) {
    const int64_t round = per_cu * dev.cus;
    if (2 * base <= round)
      splits = (int)std::max<int64_t>(1, std::min<int64_t>(round / base, bins_per_group));
  } else {
    const int64_t target = 2 * per_cu * dev.cus;
    if (base < target) {
      int64_t want = (target + base - 1) / base;
      const int64_t step = 8 / std::gcd(G, 8);
      want = (want + step - 1) / step * step;
      const int64_t fine = std::min<int64_t>(128, bins_per_group / (8 * waves)) / step * step;
      want = std::max(want, fine);
      splits = (int)std::max<int64_t>(1, std::min<int64_t>(want, bins_per_group));
    }
  }
  plan.RW = RW;
  plan.waves = waves;
  plan.priv = priv;
  plan.sx = sx;
  plan.sp = sp;
  plan.width = width;
  plan.lds = lds;
  plan.splits = splits;
  plan.tiles = tiles;
  return GTS_OK;
}

template <typename T, bool INTER>
gts_status launch(const gts_model* m, const void* blob, const float* X, int64_t rows, int64_t ld,
                  void* phi, hipStream_t stream) {
  Plan plan;
  const gts_status st = plan_launch<T, INTER>(m, rows, device_info(), plan);
  if (st != GTS_OK) return st;
  const int RW = plan.RW, waves = plan.waves, splits = plan.splits;
  const int32_t sx = plan.sx, sp = plan.sp, width = plan.width;
  const size_t lds = plan.lds;
#define GTS_LAUNCH(rw, w)                                                                 \
  return launch_rw<T, rw, INTER, w, false>(m, blob, X, rows, ld, phi, stream, splits, sx, sp, \
                                           width, lds)
  if (plan.priv)
    return launch_rw<T, 64, INTER, 4, true>(m, blob, X, rows, ld, phi, stream, splits, sx, sp,
                                            width, lds);
  switch (RW) {
    case 64: GTS_LAUNCH(64, 8);
    case 32: GTS_LAUNCH(32, 8);
    case 16:
      if (waves == 12) GTS_LAUNCH(16, 12);
      if (waves == 16) GTS_LAUNCH(16, 16);
      GTS_LAUNCH(16, 8);
    case 8:
      if (waves == 12) GTS_LAUNCH(8, 12);
      if (waves == 16) GTS_LAUNCH(8, 16);
      GTS_LAUNCH(8, 8);
    default:
      if (waves == 12) GTS_LAUNCH(4, 12);
      if (waves == 16) GTS_LAUNCH(4, 16);
      GTS_LAUNCH(4, 8);
  }
#undef GTS_LAUNCH
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
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (model->dtype == GTS_F64)
    return inter ? launch<double, true>(model, d_model, d_X, rows, ld_x, d_phi, s)
                 : launch<double, false>(model, d_model, d_X, rows, ld_x, d_phi, s);
  return inter ? launch<float, true>(model, d_model, d_X, rows, ld_x, d_phi, s)
               : launch<float, false>(model, d_model, d_X, rows, ld_x, d_phi, s);
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
