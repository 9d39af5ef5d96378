// Device half of libgts for gfx950 (CDNA4, wave64): SHAP values and SHAP
// interaction values of merged tree paths.
//
// Mapping ("row-lane").  A lane owns one (row, path) pair and runs the whole
// per-path dynamic programme of Algorithm 1 in its registers; a wave holds RW
// rows x (64/RW) paths.  Paths are visited in groups of equal length (the
// model layout sorts them), so the trip counts are compile-time constants and
// a wave never diverges on path length.  With RW == 64 every lane of a wave
// shares one path, whose elements are then read with scalar loads.
//
// Arithmetic.  EXTEND (Algorithm 1) keeps permutation weights w_k that are
// the polynomial coefficients E_k of prod_k (z_k + o_k t) scaled by
// k!(l-k)!/(l+1)!.  The kernels keep E_k itself: adding an element is then
// E_k <- z E_k + o E_{k-1} (one multiply-add), and the scale factors move
// into the final sum as the Shapley weights c_k = k!(q-1-k)!/q!.  UNWIND of
// element i (o_i = 1) divides the polynomial by (z_i + t) from the top
// coefficient down, as Algorithm 1's o != 0 branch does; for o_i = 0 the
// contribution reduces to -v * sum_k c_k E_k, the same for every such
// element, so no division by a zero fraction ever happens.
//
// Accumulation.  A workgroup owns a tile of RW rows for one output group and
// a slice of that group's paths; contributions go to a phi tile in LDS with
// LDS atomics and the tile is written (or atomically added, when the path
// list is split across workgroups) to HBM once.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdio>
#include <mutex>
#include <vector>

#include "gts_internal.h"

namespace gts {
namespace {

constexpr int kWaves = 4;              // waves per workgroup
constexpr int kBlock = 64 * kWaves;    // threads per workgroup
constexpr int kMaxUnrolledShap = 16;   // longest path (features) with unrolled code
constexpr int kMaxUnrolledInter = 8;

template <typename T>
struct DevModel {
  const int32_t* __restrict__ feat;
  const float* __restrict__ lower;
  const float* __restrict__ upper;
  const T* __restrict__ zero;
  const int32_t* __restrict__ path_first;
  const int32_t* __restrict__ path_len;
  const T* __restrict__ path_v;
  const int32_t* __restrict__ group_paths;
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
  d.path_first = reinterpret_cast<const int32_t*>(b + m->off[kPathFirst]);
  d.path_len = reinterpret_cast<const int32_t*>(b + m->off[kPathLen]);
  d.path_v = reinterpret_cast<const T*>(b + m->off[kPathV]);
  d.group_paths = reinterpret_cast<const int32_t*>(b + m->off[kGroupPaths]);
  d.bias = reinterpret_cast<const T*>(b + m->off[kBias]);
  d.M = m->num_features;
  d.G = m->num_groups;
  return d;
}

// Shapley weight of a coalition of size k among the other n-1 players.
__host__ __device__ constexpr double shapley_weight(int n, int k) {
  double w = 1.0;
  // k! (n-1-k)! / n!  =  1 / (n * C(n-1, k))
  double c = 1.0;
  for (int i = 1; i <= k; ++i) c = c * (double)(n - i) / (double)i;
  w = 1.0 / ((double)n * c);
  return w;
}

struct Launch {
  int64_t rows;
  int64_t ld;
  int32_t row_tiles;
  int32_t splits;   // path-list slices per group
  int32_t sx;       // LDS row stride of the X tile (floats)
  int32_t sp;       // LDS row stride of the phi tile (elements)
  int32_t width;    // phi entries per (row, group): M+1 or (M+1)^2
  int32_t accumulate;  // 1: atomically add the tile to phi (phi pre-zeroed)
};

// ---------------------------------------------------------------------------
// element fetch: x value test and zero fraction of the lane's path elements
// ---------------------------------------------------------------------------

template <typename T, int Q, bool UNIFORM>
__device__ __forceinline__ void load_elements(const DevModel<T>& d, int first, int q,
                                              const float* __restrict__ xrow, int (&f)[Q],
                                              bool (&o)[Q], T (&z)[Q]) {
#pragma unroll
  for (int k = 0; k < Q; ++k) {
    if (UNIFORM || k < q) {
      const int e = first + k;
      f[k] = d.feat[e];
      const float x = xrow[f[k]];
      o[k] = (d.lower[e] <= x) && (x < d.upper[e]);
      z[k] = d.zero[e];
    } else {  // padding element: present with probability 1, changes nothing
      f[k] = -1;
      o[k] = true;
      z[k] = T(1);
    }
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

// D = E / (zi + t) for a degree-Q polynomial E with E_Q known; D has Q terms.
template <typename T, int Q>
__device__ __forceinline__ void unwind_one(const T (&E)[Q + 1], T zi, T (&D)[Q]) {
  D[Q - 1] = E[Q];
#pragma unroll
  for (int k = Q - 1; k >= 1; --k) D[k - 1] = fma(-zi, D[k], E[k]);
}

// ---------------------------------------------------------------------------
// SHAP values of one (row, path) per lane, Q features per path
// ---------------------------------------------------------------------------

template <typename T, int Q, bool UNIFORM>
__device__ __forceinline__ void shap_round(const DevModel<T>& d, int p, bool active,
                                           const float* __restrict__ xrow, T* __restrict__ prow) {
  const int first = d.path_first[p] + 1;
  const int q = UNIFORM ? Q : d.path_len[p] - 1;
  const T v = d.path_v[p];
  int f[Q];
  bool o[Q];
  T z[Q];
  load_elements<T, Q, UNIFORM>(d, first, q, xrow, f, o, z);
  T E[Q + 1];
  extend_all<T, Q>(o, z, E);
  // shared contribution of every element with o = 0
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
    if (active && f[i] >= 0) atomicAdd(&prow[f[i]], phi);
  }
}

// Paths longer than the unrolled variants: same arithmetic with runtime loops,
// always in fp64.  Dividing the weight polynomial from its top coefficient
// down cancels more and more as paths grow; in fp32 the error passes the
// parity bound beyond about 20 features, in fp64 it stays far inside it for
// the longest path a wave64 holds (63 features).  FP64 FMAs run at the same
// rate as unpacked FP32 ones on gfx950.
template <typename T>
__device__ void shap_round_dyn(const DevModel<T>& d, int p, bool active,
                               const float* __restrict__ xrow, T* __restrict__ prow) {
  const int first = d.path_first[p] + 1;
  const int q = d.path_len[p] - 1;
  const double v = (double)d.path_v[p];
  double E[kMaxPathLen];
  double z[kMaxPathLen];
  double D[kMaxPathLen];
  uint64_t obits = 0;
  E[0] = 1.0;
  for (int l = 1; l <= q; ++l) {
    const int e = first + l - 1;
    const float x = xrow[d.feat[e]];
    const bool ol = (d.lower[e] <= x) && (x < d.upper[e]);
    const double zl = (double)d.zero[e];
    z[l - 1] = zl;
    obits |= (uint64_t)ol << (l - 1);
    E[l] = ol ? E[l - 1] : 0.0;
    for (int k = l - 1; k >= 1; --k) E[k] = fma(zl, E[k], ol ? E[k - 1] : 0.0);
    E[0] = zl * E[0];
  }
  double t_all = 0.0;
  for (int k = 0; k < q; ++k) t_all = fma(shapley_weight(q, k), E[k], t_all);
  for (int i = 0; i < q; ++i) {
    D[q - 1] = E[q];
    for (int k = q - 1; k >= 1; --k) D[k - 1] = fma(-z[i], D[k], E[k]);
    double s = 0.0;
    for (int k = 0; k < q; ++k) s = fma(shapley_weight(q, k), D[k], s);
    const bool oi = (obits >> i) & 1u;
    const double phi = oi ? v * (1.0 - z[i]) * s : -v * t_all;
    if (active) atomicAdd(&prow[d.feat[first + i]], (T)phi);
  }
}

// ---------------------------------------------------------------------------
// SHAP interaction values of one (row, path) per lane
// ---------------------------------------------------------------------------
// For elements i != c of a path with value v the interaction through this
// path is Delta_ic = v/2 (o_i - z_i)(o_c - z_c) S_ic, where S_ic is the
// Shapley-weighted sum over the path without i and c (weights for q-1
// players).  By cases on (o_i, o_c):
//   (1,1): S_ic from E / ((z_i + t)(z_c + t))
//   (1,0): (o_c - z_c) S_ic = -sum_k c'_k D^i_k           (D^i = E / (z_i + t))
//   (0,0): (o_i - z_i)(o_c - z_c) S_ic = sum_k c'_k E_k
// phi_ii = phi_i - sum_{c != i} Delta_ic (Eq. 6).

template <typename T, int Q, bool UNIFORM>
__device__ __forceinline__ void inter_round(const DevModel<T>& d, int p, bool active,
                                            const float* __restrict__ xrow, T* __restrict__ prow,
                                            int stride) {
  const int first = d.path_first[p] + 1;
  const int q = UNIFORM ? Q : d.path_len[p] - 1;
  const T v = d.path_v[p];
  int f[Q];
  bool o[Q];
  T z[Q];
  load_elements<T, Q, UNIFORM>(d, first, q, xrow, f, o, z);
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
    if constexpr (Q >= 2) {
      T acc = T(0);
#pragma unroll
      for (int k = 0; k < Q - 1; ++k) acc = fma(T(shapley_weight(Q - 1, k)), D[k], acc);
      tp[c] = acc;
    } else {
      tp[c] = T(0);
    }
#pragma unroll
    for (int i = 0; i < c; ++i) {
      // (1,1): divide D^c by (z_i + t) -> Q-1 terms, weighted sum
      T DD[Q];
      if constexpr (Q >= 2) {
        DD[Q - 2] = D[Q - 1];
#pragma unroll
        for (int k = Q - 2; k >= 1; --k) DD[k - 1] = fma(-z[i], DD[k], D[k]);
      }
      T s11 = T(0);
#pragma unroll
      for (int k = 0; k < Q - 1; ++k) s11 = fma(T(shapley_weight(Q - 1, k)), DD[k], s11);
      T delta;
      if (o[i] && o[c]) delta = half_v * (T(1) - z[i]) * (T(1) - z[c]) * s11;
      else if (o[i]) delta = -half_v * (T(1) - z[i]) * tp[i];
      else if (o[c]) delta = -half_v * (T(1) - z[c]) * tp[c];
      else delta = half_v * t_pair;
      diag[c] -= delta;
      diag[i] -= delta;
      if (active && f[i] >= 0 && f[c] >= 0) {
        atomicAdd(&prow[f[i] * stride + f[c]], delta);
        atomicAdd(&prow[f[c] * stride + f[i]], delta);
      }
    }
  }
#pragma unroll
  for (int c = 0; c < Q; ++c)
    if (active && f[c] >= 0) atomicAdd(&prow[f[c] * stride + f[c]], diag[c]);
}

// Long paths: runtime loops, always in fp64 (see shap_round_dyn).
template <typename T>
__device__ void inter_round_dyn(const DevModel<T>& d, int p, bool active,
                                const float* __restrict__ xrow, T* __restrict__ prow, int stride) {
  const int first = d.path_first[p] + 1;
  const int q = d.path_len[p] - 1;
  const double v = (double)d.path_v[p];
  double E[kMaxPathLen];
  double z[kMaxPathLen];
  double D[kMaxPathLen];
  double DD[kMaxPathLen];
  double tp[kMaxPathLen];
  double diag[kMaxPathLen];
  uint64_t obits = 0;
  E[0] = 1.0;
  for (int l = 1; l <= q; ++l) {
    const int e = first + l - 1;
    const float x = xrow[d.feat[e]];
    const bool ol = (d.lower[e] <= x) && (x < d.upper[e]);
    const double zl = (double)d.zero[e];
    z[l - 1] = zl;
    obits |= (uint64_t)ol << (l - 1);
    E[l] = ol ? E[l - 1] : 0.0;
    for (int k = l - 1; k >= 1; --k) E[k] = fma(zl, E[k], ol ? E[k - 1] : 0.0);
    E[0] = zl * E[0];
  }
  double t_all = 0.0, t_pair = 0.0;
  for (int k = 0; k < q; ++k) t_all = fma(shapley_weight(q, k), E[k], t_all);
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
    const int fc = d.feat[first + c];
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
      const int fi = d.feat[first + i];
      if (active) {
        atomicAdd(&prow[fi * stride + fc], (T)delta);
        atomicAdd(&prow[fc * stride + fi], (T)delta);
      }
    }
  }
  for (int c = 0; c < q; ++c)
    if (active) {
      const int fc = d.feat[first + c];
      atomicAdd(&prow[fc * stride + fc], (T)diag[c]);
    }
}

// ---------------------------------------------------------------------------
// workgroup driver
// ---------------------------------------------------------------------------

template <typename T, int RW, bool INTER>
__device__ __forceinline__ void dispatch_round(int Q, const DevModel<T>& d, int p, bool active,
                                               const float* xrow, T* prow) {
  constexpr bool U = (RW == 64);
  if constexpr (INTER) {
    switch (Q) {
#define GTS_CASE(n) case n: inter_round<T, n, U>(d, p, active, xrow, prow, d.M + 1); break;
      GTS_CASE(1) GTS_CASE(2) GTS_CASE(3) GTS_CASE(4) GTS_CASE(5) GTS_CASE(6)
      GTS_CASE(7) GTS_CASE(8)
#undef GTS_CASE
      default: inter_round_dyn<T>(d, p, active, xrow, prow, d.M + 1); break;
    }
  } else {
    switch (Q) {
#define GTS_CASE(n) case n: shap_round<T, n, U>(d, p, active, xrow, prow); break;
      GTS_CASE(1) GTS_CASE(2) GTS_CASE(3) GTS_CASE(4) GTS_CASE(5) GTS_CASE(6)
      GTS_CASE(7) GTS_CASE(8) GTS_CASE(9) GTS_CASE(10) GTS_CASE(11) GTS_CASE(12)
      GTS_CASE(13) GTS_CASE(14) GTS_CASE(15) GTS_CASE(16)
#undef GTS_CASE
      default: shap_round_dyn<T>(d, p, active, xrow, prow); break;
    }
  }
}

// One workgroup: rows [tile*RW, tile*RW + RW) of output group g, paths of
// slice s of that group.  blockIdx.x = (tile * G + g) * S + s, so with S a
// multiple of 8 each XCD (blocks are dealt round-robin to the 8 XCDs) reads
// only its own slices of the path list.
template <typename T, int RW, bool INTER>
__global__ __launch_bounds__(kBlock) void rowlane_kernel(DevModel<T> d, const float* __restrict__ X,
                                                        T* __restrict__ phi, Launch L) {
  extern __shared__ __align__(16) unsigned char smem[];
  constexpr int P = 64 / RW;  // paths per wave round
  const int M = d.M;
  const int G = d.G;
  const int64_t b = blockIdx.x;
  const int s = (int)(b % L.splits);
  const int64_t tg = b / L.splits;
  const int g = (int)(tg % G);
  const int64_t tile = tg / G;
  const int64_t r0 = tile * RW;

  float* xs = reinterpret_cast<float*>(smem);
  T* ps = reinterpret_cast<T*>(smem + (size_t)RW * L.sx * sizeof(float));

  // stage the X tile (coalesced along each row) and clear the phi tile
  for (int i = threadIdx.x; i < RW * M; i += kBlock) {
    const int r = i / M, c = i - r * M;
    const int64_t row = r0 + r;
    xs[r * L.sx + c] = row < L.rows ? X[row * L.ld + c] : 0.0f;
  }
  for (int i = threadIdx.x; i < RW * L.sp; i += kBlock) ps[i] = T(0);
  __syncthreads();

  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int r = lane % RW;
  const int j = lane / RW;
  const int g0 = d.group_paths[g], g1 = d.group_paths[g + 1];
  const int n = g1 - g0;
  int chunk = (n + L.splits - 1) / L.splits;
  chunk = (chunk + P - 1) / P * P;
  const int a = g0 + min(n, s * chunk);
  const int e = g0 + min(n, (s + 1) * chunk);
  const int rounds = (e - a + P - 1) / P;
  const float* xrow = xs + r * L.sx;
  T* prow = ps + r * L.sp;
  for (int rd = wave; rd < rounds; rd += kWaves) {
    const int lead = __builtin_amdgcn_readfirstlane(a + rd * P);
    const int Q = __builtin_amdgcn_readfirstlane(d.path_len[lead]) - 1;
    int p = lead + j;
    const bool active = p < e;
    if (!active) p = lead;
    if (RW == 64) p = __builtin_amdgcn_readfirstlane(p);
    if (Q > 0) dispatch_round<T, RW, INTER>(Q, d, p, active, xrow, prow);
  }
  __syncthreads();

  // write the tile: phi[row][g][.]; the bias goes to the last entry
  const T bias = d.bias[g];
  const int W = L.width;
  for (int i = threadIdx.x; i < RW * W; i += kBlock) {
    const int rr = i / W, c = i - rr * W;
    const int64_t row = r0 + rr;
    if (row >= L.rows) continue;
    T val = ps[rr * L.sp + c];
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

int device_cus() {
  static std::mutex mu;
  static std::vector<int> cus;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 256;
  std::lock_guard<std::mutex> lock(mu);
  if ((int)cus.size() <= dev) cus.resize(dev + 1, 0);
  if (cus[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
      n = 256;
    cus[dev] = n;
  }
  return cus[dev];
}

constexpr int64_t kLdsBudget = 64 * 1024;

inline int odd_at_least(int n) { return n | 1; }

template <typename T, int RW, bool INTER>
gts_status launch_rw(const gts_model* m, const void* blob, const float* X, int64_t rows,
                     int64_t ld, void* phi, hipStream_t stream, int splits, int32_t sx, int32_t sp,
                     int32_t width, size_t lds) {
  DevModel<T> d = dev_model<T>(m, blob);
  Launch L;
  L.rows = rows;
  L.ld = ld;
  L.row_tiles = (int32_t)((rows + RW - 1) / RW);
  L.splits = splits;
  L.sx = sx;
  L.sp = sp;
  L.width = width;
  L.accumulate = splits > 1 ? 1 : 0;
  const int64_t total = (int64_t)rows * m->num_groups * width;
  if (L.accumulate) {
    const int64_t blocks = std::min<int64_t>((total + 255) / 256, 65536);
    hipLaunchKernelGGL(fill_zero<T>, dim3((unsigned)blocks), dim3(256), 0, stream,
                       static_cast<T*>(phi), total);
  }
  const int64_t grid = (int64_t)L.row_tiles * m->num_groups * splits;
  if (grid > 0x7fffffffLL) return fail(GTS_EINVAL, "problem too large for one launch");
  auto kern = rowlane_kernel<T, RW, INTER>;
  if (lds > 48 * 1024) {
    if (hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) != hipSuccess)
      return fail(GTS_EDEVICE, "cannot raise the LDS limit to %zu bytes", lds);
  }
  hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(kBlock), lds, stream, d, X,
                     static_cast<T*>(phi), L);
  const hipError_t err = hipGetLastError();
  if (err != hipSuccess) return fail(GTS_EDEVICE, "kernel launch failed: %s", hipGetErrorString(err));
  return GTS_OK;
}

template <typename T, bool INTER>
gts_status launch(const gts_model* m, const void* blob, const float* X, int64_t rows, int64_t ld,
                  void* phi, hipStream_t stream) {
  const int M = m->num_features;
  const int G = m->num_groups;
  const int32_t width = INTER ? (M + 1) * (M + 1) : (M + 1);
  const int32_t sx = odd_at_least(M);
  const int32_t sp = odd_at_least(width);
  // largest row tile whose X and phi tiles fit the LDS budget
  int RW = 0;
  size_t lds = 0;
  for (int cand : {64, 32, 16, 8, 4}) {
    const size_t need = (size_t)cand * ((size_t)sx * sizeof(float) + (size_t)sp * sizeof(T));
    if ((int64_t)need <= kLdsBudget) { RW = cand; lds = need; break; }
  }
  if (RW == 0)
    return fail(GTS_EINVAL, "M = %d is too large for an LDS tile of 4 rows", M);
  // enough workgroups to give every CU several; slices a multiple of 8 (XCDs)
  const int64_t tiles = (rows + RW - 1) / RW;
  const int64_t base = tiles * G;
  const int64_t target = 8LL * device_cus();
  int splits = 1;
  if (base < target) {
    const int64_t max_paths = std::max<int64_t>(1, m->num_paths / G);
    splits = (int)std::min<int64_t>((target + base - 1) / base, max_paths / (64 / RW) + 1);
    splits = std::max(1, splits);
    if (splits > 1) splits = (splits + 7) / 8 * 8;
  }
  switch (RW) {
    case 64: return launch_rw<T, 64, INTER>(m, blob, X, rows, ld, phi, stream, splits, sx, sp, width, lds);
    case 32: return launch_rw<T, 32, INTER>(m, blob, X, rows, ld, phi, stream, splits, sx, sp, width, lds);
    case 16: return launch_rw<T, 16, INTER>(m, blob, X, rows, ld, phi, stream, splits, sx, sp, width, lds);
    case 8: return launch_rw<T, 8, INTER>(m, blob, X, rows, ld, phi, stream, splits, sx, sp, width, lds);
    default: return launch_rw<T, 4, INTER>(m, blob, X, rows, ld, phi, stream, splits, sx, sp, width, lds);
  }
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
