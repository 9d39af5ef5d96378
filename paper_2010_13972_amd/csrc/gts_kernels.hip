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
// compile-time constants (one variant per path length up to 16 features, 8
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
// Algorithm 1's o != 0 branch; for o = 0 the contribution reduces to
// -v * sum_k c_k E_k, shared by every such element, so no division by a zero
// fraction is ever needed.
//
// Accumulation.  A workgroup owns a tile of RW rows of one output group and a
// slice of that group's bins.  Contributions go to a phi tile in LDS (an
// atomic add built from compare-and-swap); the tile is written to HBM once
// (atomically added when several workgroups share the row tile).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <mutex>
#include <numeric>
#include <vector>

#include "gts_internal.h"

namespace gts {
namespace {

constexpr int kMaxUnrolledShap = 16;   // longest path (features) with unrolled code
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

// Accumulate into the phi tile.  EXCL: no other lane or wave can update the
// same entry at the same time (a wave-private tile with one path per wave),
// so a plain read-modify-write suffices.
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

// One wave's copy of its current bin in LDS: element e (a lane of the bin)
// as (feature, lower, upper, zero fraction or leaf value).  Paths start at a
// table built from the root ballot: start[t] = bin lane of the t-th root,
// start[#roots] = bin length.
template <typename T>
struct Stage {
  int4 meta[64];   // feature, lower bits, upper bits, z bits (fp32 z only)
  T zd[64];        // z in the model dtype
  int start[65];
};

template <typename T>
__device__ __forceinline__ int stage_bin(Stage<T>* st, const Bin<T>& b, int lane) {
  st->meta[lane] = make_int4(b.feat, __float_as_int(b.lo), __float_as_int(b.hi),
                             sizeof(T) == 4 ? __float_as_int((float)b.z) : 0);
  st->zd[lane] = b.z;
  const bool root = b.feat == -1;
  const uint64_t roots = __ballot(root);
  const int rank = __builtin_amdgcn_mbcnt_hi((unsigned)(roots >> 32),
                                             __builtin_amdgcn_mbcnt_lo((unsigned)roots, 0u));
  if (root) st->start[rank] = lane;
  const int nroots = __popcll(roots);
  if (lane == 0) st->start[nroots] = b.len;
  // the stores above are read by other lanes of this wave only
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  return nroots;
}

// Element k (0-based among the path's features) of the path whose root is
// at bin lane s; s is wave-uniform when one path fills the wave.
template <typename T>
struct Fetch {
  const Stage<T>* st;
  int s;
  __device__ __forceinline__ void get(int k, int& f, float& lo, float& hi, T& z) const {
    const int e = (s + 1 + k) & 63;
    const int4 m = st->meta[e];
    f = m.x;
    lo = __int_as_float(m.y);
    hi = __int_as_float(m.z);
    if constexpr (sizeof(T) == 4) z = __int_as_float(m.w);
    else z = st->zd[e];
  }
  __device__ __forceinline__ T v() const {
    if constexpr (sizeof(T) == 4) return __int_as_float(st->meta[s & 63].w);
    else return st->zd[s & 63];
  }
};

// Feature, presence test o_k = [lower <= x < upper] and zero fraction of
// the first Q elements.  Elements k >= q are padding: present with
// probability 1 and absent with probability 1 (z = o = 1), which changes no
// other element's Shapley value; f = -1 marks them unwritten.
template <typename T, int Q, bool UNIFORM>
__device__ __forceinline__ void load_path(const Fetch<T>& fe, int q, const float* __restrict__ xrow,
                                          int (&f)[Q], bool (&o)[Q], T (&z)[Q]) {
#pragma unroll
  for (int k = 0; k < Q; ++k) {
    int fk;
    float lo, hi;
    T zk;
    fe.get(k, fk, lo, hi, zk);
    const bool real = UNIFORM || k < q;
    const float x = xrow[real ? fk : 0];
    f[k] = real ? fk : -1;
    o[k] = real ? (lo <= x) && (x < hi) : true;
    z[k] = real ? zk : T(1);
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

// SHAP values: phi[f_i] += v (o_i - z_i) * sum_k c_k D^i_k
template <typename T, int Q, bool EXCL>
__device__ __forceinline__ void shap_math(const int (&f)[Q], const bool (&o)[Q], const T (&z)[Q],
                                          T v, bool active, T* __restrict__ prow) {
  T E[Q + 1];
  extend_all<T, Q>(o, z, E);
  T t_all = T(0);
#pragma unroll
  for (int k = 0; k < Q; ++k) t_all = fma(T(shapley_weight(Q, k)), E[k], t_all);
  const T neg_vt = -v * t_all;
#pragma unroll
  for (int i = 0; i < Q; ++i) {
    T D[Q];
    unwind_one<T, Q>(E, z[i], D);
    T s = T(0);
#pragma unroll
    for (int k = 0; k < Q; ++k) s = fma(T(shapley_weight(Q, k)), D[k], s);
    const T phi = o[i] ? v * (T(1) - z[i]) * s : neg_vt;
    if (active && f[i] >= 0) acc_add<EXCL>(&prow[f[i]], phi);
  }
}

// Interaction values.  For elements i != c the interaction through this path
// is Delta_ic = v/2 (o_i - z_i)(o_c - z_c) S_ic, S_ic the Shapley-weighted sum
// over the path without i and c (weights for q-1 players).  By cases on
// (o_i, o_c):
//   (1,1): S_ic from E / ((z_i + t)(z_c + t))
//   (1,0): (o_c - z_c) S_ic = -sum_k c'_k D^i_k         (D^i = E / (z_i + t))
//   (0,0): (o_i - z_i)(o_c - z_c) S_ic = sum_k c'_k E_k
// and phi_ii = phi_i - sum_{c != i} Delta_ic (Eq. 6).
template <typename T, int Q, bool EXCL>
__device__ __forceinline__ void inter_math(const int (&f)[Q], const bool (&o)[Q], const T (&z)[Q],
                                           T v, bool active, T* __restrict__ prow, int stride) {
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
  T tp[Q];    // sum_k c'_k D^c_k for each element c
  T diag[Q];  // running phi_cc
#pragma unroll
  for (int c = 0; c < Q; ++c) {
    T D[Q];
    unwind_one<T, Q>(E, z[c], D);
    T s = T(0);
#pragma unroll
    for (int k = 0; k < Q; ++k) s = fma(T(shapley_weight(Q, k)), D[k], s);
    diag[c] = o[c] ? v * (T(1) - z[c]) * s : -v * t_all;
    tp[c] = T(0);
    if constexpr (Q >= 2) {
#pragma unroll
      for (int k = 0; k < Q - 1; ++k) tp[c] = fma(T(shapley_weight(Q - 1, k)), D[k], tp[c]);
    }
#pragma unroll
    for (int i = 0; i < c; ++i) {
      T s11 = T(0);
      if constexpr (Q >= 2) {
        T DD[Q];
        DD[Q - 2] = D[Q - 1];
#pragma unroll
        for (int k = Q - 2; k >= 1; --k) DD[k - 1] = fma(-z[i], DD[k], D[k]);
#pragma unroll
        for (int k = 0; k < Q - 1; ++k) s11 = fma(T(shapley_weight(Q - 1, k)), DD[k], s11);
      }
      T delta;
      if (o[i] && o[c]) delta = half_v * (T(1) - z[i]) * (T(1) - z[c]) * s11;
      else if (o[i]) delta = -half_v * (T(1) - z[i]) * tp[i];
      else if (o[c]) delta = -half_v * (T(1) - z[c]) * tp[c];
      else delta = half_v * t_pair;
      diag[c] -= delta;
      diag[i] -= delta;
      if (active && f[i] >= 0 && f[c] >= 0) {
        acc_add<EXCL>(&prow[f[i] * stride + f[c]], delta);
        acc_add<EXCL>(&prow[f[c] * stride + f[i]], delta);
      }
    }
  }
#pragma unroll
  for (int c = 0; c < Q; ++c)
    if (active && f[c] >= 0) acc_add<EXCL>(&prow[f[c] * stride + f[c]], diag[c]);
}

// Paths longer than the unrolled variants: the same arithmetic with runtime
// loops, always in fp64.  Dividing the weight polynomial from its top
// coefficient down cancels more and more as paths grow; in fp32 the error
// passes the parity bound beyond about 20 features, in fp64 it stays far
// inside it for the longest path a wave64 holds (63 features).  FP64 FMAs run
// at the rate of unpacked FP32 ones on gfx950.
template <typename T, bool INTER, bool EXCL>
__device__ void path_dyn(const Fetch<T>& fe, int qfetch, int q, bool active,
                         const float* __restrict__ xrow, T* __restrict__ prow, int stride) {
  double E[kMaxPathLen];
  double z[kMaxPathLen];
  double D[kMaxPathLen];
  int f[kMaxPathLen];
  uint64_t obits = 0;
  for (int k = 0; k < qfetch; ++k) {
    int fk;
    float lo, hi;
    T zt;
    fe.get(k, fk, lo, hi, zt);
    const double zk = (double)zt;
    if (k < q) {
      const float x = xrow[fk];
      f[k] = fk;
      z[k] = zk;
      obits |= (uint64_t)((lo <= x) && (x < hi)) << k;
    }
  }
  const double v = (double)fe.v();
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
      if (active) acc_add<EXCL>(&prow[f[i]], (T)phi);
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
        if (active) {
          acc_add<EXCL>(&prow[f[i] * stride + f[c]], (T)delta);
          acc_add<EXCL>(&prow[f[c] * stride + f[i]], (T)delta);
        }
      }
    }
    for (int c = 0; c < q; ++c)
      if (active) acc_add<EXCL>(&prow[f[c] * stride + f[c]], (T)diag[c]);
  }
}

template <typename T, int Q, bool UNIFORM, bool INTER, bool EXCL>
__device__ __forceinline__ void path_fixed(const Fetch<T>& fe, int q, bool active,
                                           const float* __restrict__ xrow, T* __restrict__ prow,
                                           int stride) {
  int f[Q];
  bool o[Q];
  T z[Q];
  load_path<T, Q, UNIFORM>(fe, q, xrow, f, o, z);
  const T v = fe.v();
  if constexpr (INTER) inter_math<T, Q, EXCL>(f, o, z, v, active, prow, stride);
  else shap_math<T, Q, EXCL>(f, o, z, v, active, prow);
}

// Q = features of the longest path in the wave's current set (uniform)
template <typename T, bool UNIFORM, bool INTER, bool EXCL>
__device__ __forceinline__ void dispatch(int Q, const Fetch<T>& fe, int q, bool active,
                                         const float* xrow, T* prow, int stride) {
  static_assert(kMaxUnrolledShap == 16 && kMaxUnrolledInter == 8, "update the case lists");
  if constexpr (INTER) {
    switch (Q) {
#define GTS_CASE(n) case n: path_fixed<T, n, UNIFORM, true, EXCL>(fe, q, active, xrow, prow, stride); break;
      GTS_CASE(1) GTS_CASE(2) GTS_CASE(3) GTS_CASE(4) GTS_CASE(5) GTS_CASE(6)
      GTS_CASE(7) GTS_CASE(8)
#undef GTS_CASE
      default: path_dyn<T, true, EXCL>(fe, Q, q, active, xrow, prow, stride); break;
    }
  } else {
    switch (Q) {
#define GTS_CASE(n) case n: path_fixed<T, n, UNIFORM, false, EXCL>(fe, q, active, xrow, prow, stride); break;
      GTS_CASE(1) GTS_CASE(2) GTS_CASE(3) GTS_CASE(4) GTS_CASE(5) GTS_CASE(6)
      GTS_CASE(7) GTS_CASE(8) GTS_CASE(9) GTS_CASE(10) GTS_CASE(11) GTS_CASE(12)
      GTS_CASE(13) GTS_CASE(14) GTS_CASE(15) GTS_CASE(16)
#undef GTS_CASE
      default: path_dyn<T, false, EXCL>(fe, Q, q, active, xrow, prow, stride); break;
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
__device__ __forceinline__ void process_bin(Stage<T>* st, const Bin<T>& b, int lane,
                                            const float* xrow, T* prow, int stride) {
  const int nroots = stage_bin(st, b, lane);
  if constexpr (RW == 64) {
    for (int t = 0; t < nroots; ++t) {
      const int s = __builtin_amdgcn_readfirstlane(st->start[t]);
      const int q = __builtin_amdgcn_readfirstlane(st->start[t + 1]) - s - 1;
      if (q > 0) dispatch<T, true, INTER, EXCL>(q, Fetch<T>{st, s}, q, true, xrow, prow, stride);
    }
  } else {
    constexpr int P = 64 / RW;
    const int j = lane / RW;
    for (int base = 0; base < nroots; base += P) {
      const int t = base + j;
      const bool valid = t < nroots;
      const int my_s = valid ? st->start[t] : 0;
      const int my_q = valid ? st->start[t + 1] - my_s - 1 : 0;
      const int qmax = wave_max_small(my_q);
      if (qmax > 0)
        dispatch<T, false, INTER, false>(qmax, Fetch<T>{st, my_s}, my_q, my_q > 0, xrow, prow, stride);
    }
  }
  // the next bin overwrites the stage
  __builtin_amdgcn_wave_barrier();
}

// One workgroup: rows [tile*RW, tile*RW + RW) of output group g, bins of
// slice s of that group.  PRIV: every wave accumulates into a phi tile of its
// own (summed when the tile is written), so waves never contend; with one
// path per wave (RW == 64) the accumulation then needs no atomics.
// Workgroups are dealt to the 8 XCDs round-robin; when the (group, slice)
// units divide evenly among the XCDs, consecutive workgroups on an XCD take
// the same unit for successive row tiles, so each XCD's L2 holds only its own
// part of the model.
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
  Stage<T>* stages = reinterpret_cast<Stage<T>*>(
      smem + (((size_t)RW * L.sx * sizeof(float) + (size_t)NT * tile_elems * sizeof(T) + 15) & ~(size_t)15));

  // stage the X tile (coalesced along each row) and clear the phi tile
  for (int i = threadIdx.x; i < RW * M; i += kThreads) {
    const int r = i / M, c = i - r * M;
    const int64_t row = r0 + r;
    xs[r * L.sx + c] = row < L.rows ? X[row * L.ld + c] : 0.0f;
  }
  for (int i = threadIdx.x; i < NT * tile_elems; i += kThreads) ps[i] = T(0);
  __syncthreads();

  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int r = lane % RW;
  const int gb0 = d.group_bins[g], gb1 = d.group_bins[g + 1];
  const int nb = gb1 - gb0;
  const int chunk = (nb + L.splits - 1) / L.splits;
  const int b_lo = gb0 + min(nb, s * chunk);
  const int b_hi = gb0 + min(nb, (s + 1) * chunk);
  const float* xrow = xs + r * L.sx;
  T* prow = ps + (PRIV ? wave * tile_elems : 0) + r * L.sp;
  const int stride = M + 1;

  int bi = b_lo + wave;
  if (bi < b_hi) {
    Bin<T> cur = load_bin(d, bi, lane);
    for (; bi < b_hi; bi += WAVES) {
      Bin<T> nxt;
      const int bn = bi + WAVES;
      if (bn < b_hi) nxt = load_bin(d, bn, lane);
      process_bin<T, RW, INTER, PRIV && RW == 64>(stages + wave, cur, lane, xrow, prow, stride);
      cur = nxt;
    }
  }
  __syncthreads();

  // write the tile: phi[row][g][.]; the bias goes to the last entry
  const T bias = d.bias[g];
  const int W = L.width;
  for (int i = threadIdx.x; i < RW * W; i += kThreads) {
    const int rr = i / W, c = i - rr * W;
    const int64_t row = r0 + rr;
    if (row >= L.rows) continue;
    T val = ps[rr * L.sp + c];
#pragma unroll
    for (int w = 1; w < NT; ++w) val += ps[w * tile_elems + rr * L.sp + c];
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

template <typename T, bool INTER>
gts_status launch(const gts_model* m, const void* blob, const float* X, int64_t rows, int64_t ld,
                  void* phi, hipStream_t stream) {
  const DeviceInfo dev = device_info();
  const int M = m->num_features;
  const int G = m->num_groups;
  const int64_t width64 = INTER ? (int64_t)(M + 1) * (M + 1) : (int64_t)(M + 1);
  if (width64 > (1 << 30)) return fail(GTS_EINVAL, "M = %d is too large", M);
  const int32_t width = (int32_t)width64;
  const int32_t sx = odd_at_least(M);
  const int32_t sp = odd_at_least(width);
  // Row tile and accumulation.  If 64 rows with a private phi tile for each
  // of 4 waves fit in 64 KB, use them (no contention, no atomics).  Otherwise
  // 8 waves share one tile: the largest RW whose tiles fit in 64 KB (several
  // workgroups per CU), or, if that would leave fewer than 8 rows per wave,
  // 8 rows (then 4) using up to the whole LDS of a workgroup.
  auto need = [&](int rw, int waves, bool priv) {
    const size_t tiles = (size_t)rw * ((size_t)sx * sizeof(float) +
                                       (priv ? (size_t)waves : 1) * (size_t)sp * sizeof(T));
    return ((tiles + 15) & ~(size_t)15) + (size_t)waves * sizeof(Stage<T>);
  };
  int RW = 0;
  int waves = 8;
  bool priv = false;
  if (need(64, 4, true) <= 64 * 1024) {
    RW = 64;
    waves = 4;
    priv = true;
  } else {
    for (int cand : {64, 32, 16, 8}) {
      if (need(cand, 8, false) <= 64 * 1024) {
        RW = cand;
        break;
      }
    }
    if (RW == 0 && (int64_t)need(8, 8, false) <= dev.lds_per_block) RW = 8;
    if (RW == 0 && (int64_t)need(4, 8, false) <= dev.lds_per_block) RW = 4;
  }
  if (RW == 0) return fail(GTS_EINVAL, "M = %d needs more LDS than a workgroup has", M);
  const size_t lds = need(RW, waves, priv);
  // enough workgroups for two rounds of every CU at the occupancy the LDS
  // allows; (group, slice) units a multiple of the 8 XCDs when split
  const int64_t tiles = (rows + RW - 1) / RW;
  const int64_t base = tiles * G;
  const int64_t per_cu = std::max<int64_t>(1, std::min<int64_t>(8, dev.lds_per_cu / (int64_t)lds));
  const int64_t target = 2 * per_cu * dev.cus;
  const int64_t bins_per_group = std::max<int64_t>(1, m->num_bins / G);
  int splits = 1;
  if (base < target) {
    int64_t want = (target + base - 1) / base;
    const int64_t step = 8 / std::gcd(G, 8);
    want = (want + step - 1) / step * step;
    splits = (int)std::max<int64_t>(1, std::min<int64_t>(want, bins_per_group));
  }
#define GTS_LAUNCH(rw)                                                                    \
  return launch_rw<T, rw, INTER, 8, false>(m, blob, X, rows, ld, phi, stream, splits, sx, sp, \
                                           width, lds)
  if (priv)
    return launch_rw<T, 64, INTER, 4, true>(m, blob, X, rows, ld, phi, stream, splits, sx, sp,
                                            width, lds);
  switch (RW) {
    case 64: GTS_LAUNCH(64);
    case 32: GTS_LAUNCH(32);
    case 16: GTS_LAUNCH(16);
    case 8: GTS_LAUNCH(8);
    default: GTS_LAUNCH(4);
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

extern "C" gts_status gts_shap(const gts_model* model, const void* d_model, const float* d_X,
                               int64_t rows, int64_t ld_x, void* d_phi, void* stream) {
  return gts::entry(model, d_model, d_X, rows, ld_x, d_phi, stream, false);
}

extern "C" gts_status gts_shap_interactions(const gts_model* model, const void* d_model,
                                            const float* d_X, int64_t rows, int64_t ld_x,
                                            void* d_phi, void* stream) {
  return gts::entry(model, d_model, d_X, rows, ld_x, d_phi, stream, true);
}
