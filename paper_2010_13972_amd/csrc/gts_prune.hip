// Batch pruning of a packed model: gts_prune_workspace_bytes and
// gts_prune_model.
//
// A (row, path) pair whose path has an element of zero fraction with a range
// that misses the row's value contributes exactly nothing (Algorithm 1 prunes
// such zero-cover subtrees).  If no row of a batch has its value inside that
// range, the path contributes nothing to any row of the batch and can be left
// out of every launch for it.  This pre-pass finds those paths on the device
// and writes the others into a new blob in the caller's workspace, where
// gts_shap and gts_shap_interactions run on them as on any packed model:
//   1. sort_keys: per feature and chunk of up to 16384 rows, the rows'
//      ordered keys in ascending order (a bitonic network, 16 keys per thread
//      in registers, exchanges between threads through LDS);
//   2. mark_paths: one wave per bin, one element per lane; every
//      zero-fraction element searches its feature's sorted keys for a key in
//      its range, and a path with an element that finds none is dropped.  Each
//      kept path gets a rank among the kept paths of its output group and
//      length (one atomic add per wave and length, on one of 64 partial
//      counters);
//   3. plan_pruned: one workgroup turns the counts into bins (a block-wide
//      scan over the classes): per group, the lengths from longest to
//      shortest, each length in bins of 64 / length paths (every bin holds
//      paths of one length, so the sorted-bins flag holds), and writes the bin
//      starts, the group ranges and the bias;
//   4. copy_paths: one wave per bin again, every kept path's elements to
//      their place, unchanged (zero-fraction elements still first).
// The outcome of the test is the kernels' own range test on the same keys, so
// exactly the paths that contribute nothing to any row are dropped.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <climits>
#include <cstdint>

#include "gts_launch.h"
#include "gts_shap_kernel.h"

namespace gts {
namespace {

constexpr int kSizes = kMaxPathLen + 1;   // path lengths in elements, root included
constexpr int kParts = 64;                // partial counters per (group, length)
constexpr int kMarkWaves = 4;             // bins (waves) per workgroup of mark and copy
constexpr int kSortThreads = 1024;        // threads of a key-sorting workgroup

// Byte layout of the workspace, and of the pruned blob inside it.
struct PruneLayout {
  int64_t chunk = 1;    // keys per sorted chunk (1024 E, E = 1, 2, 4, 8 or 16)
  int64_t chunks = 0;
  int64_t keys = 0;     // int32[M][chunks][chunk]
  int64_t counts = 0;   // int32[G][kSizes][kParts]: counts, then element bases
  int64_t totals = 0;   // int32[G][kSizes][2]: paths, then element base / bin base
  int64_t ranks = 0;    // int32[num_elements]: on a root, its rank (-1: dropped)
  int64_t blob = 0;     // the pruned blob
  int64_t blob_bytes = 0;
  int64_t bytes = 0;
  int64_t off[kBlobArrays] = {};
};

int64_t aligned(int64_t n) { return (n + kBlobAlign - 1) / kBlobAlign * kBlobAlign; }

int lds_per_block() {
  int dev = 0, n = 0;
  if (hipGetDevice(&dev) == hipSuccess &&
      hipDeviceGetAttribute(&n, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) == hipSuccess &&
      n > 0)
    return n;
  return 64 * 1024;
}

PruneLayout prune_layout(const gts_model* m, int64_t rows, int lds) {
  PruneLayout L;
  // 1024 E rows per sorted chunk, E a power of two up to 16 that the LDS of
  // a workgroup holds
  int64_t cap = kSortThreads * 16;
  while (cap * (int64_t)sizeof(int32_t) > lds && cap > kSortThreads) cap >>= 1;
  L.chunk = kSortThreads;
  while (L.chunk < rows && L.chunk < cap) L.chunk <<= 1;
  L.chunks = rows > 0 ? (rows + L.chunk - 1) / L.chunk : 0;
  auto take = [&](int64_t n) {
    const int64_t o = L.bytes;
    L.bytes += aligned(n);
    return o;
  };
  const int64_t G = m->num_groups, E = m->num_elements, P = m->num_paths;
  L.keys = take((int64_t)m->num_features * L.chunks * L.chunk * (int64_t)sizeof(int32_t));
  L.counts = take(G * kSizes * kParts * (int64_t)sizeof(int32_t));
  L.totals = take(G * kSizes * 2 * (int64_t)sizeof(int32_t));
  L.ranks = take(std::max<int64_t>(E, 1) * (int64_t)sizeof(int32_t));
  const int64_t zb = m->dtype == GTS_F64 ? 8 : 4;
  int64_t o = 0;
  auto put = [&](int a, int64_t n) {
    L.off[a] = o;
    o += aligned(n);
  };
  put(kFeat, 4 * E);
  put(kLower, 4 * E);
  put(kUpper, 4 * E);
  put(kZero, zb * E);
  put(kBinStart, 4 * (P + 1));   // at most one bin per kept path
  put(kGroupBins, 4 * (G + 1));
  put(kBias, zb * G);
  L.blob = L.bytes;
  L.blob_bytes = o;
  L.bytes += o;
  return L;
}

// Bitonic stages j = J, J/2, ..., 1 of merge size k among the E keys a thread
// holds (positions pos0 .. pos0 + E - 1); stages with j >= k are not part of
// this merge and are skipped.
template <int E, int J>
__device__ __forceinline__ void register_stages(int (&v)[E], int pos0, int k) {
  if constexpr (J >= 1) {
    if (J < k) {
#pragma unroll
      for (int i = 0; i < E; ++i) {
        if ((i & J) == 0) {
          const bool up = ((pos0 + i) & k) == 0;
          const int a = v[i], b = v[i ^ J];
          v[i] = up ? min(a, b) : max(a, b);
          v[i ^ J] = up ? max(a, b) : min(a, b);
        }
      }
    }
    register_stages<E, J / 2>(v, pos0, k);
  }
}

// One workgroup of 1024 threads per (feature, chunk of 1024 E rows): the
// chunk's row keys in ascending order, by a bitonic network.  Thread t holds
// the keys of positions t E .. t E + E - 1 in registers; a stage whose
// partners are E or more positions apart exchanges them through LDS, slot i
// of thread t at i * 1024 + t (consecutive lanes, consecutive banks).  Slots
// past the chunk's last row hold INT_MAX and are never searched.

template <int E>
__global__ __launch_bounds__(kSortThreads) void sort_keys(const float* __restrict__ X,
                                                          int64_t rows, int64_t ld, int M,
                                                          int chunks, int* __restrict__ keys) {
  constexpr int N = kSortThreads * E;
  extern __shared__ int sk[];
  const int f = blockIdx.x % M;
  const int c = blockIdx.x / M;
  const int64_t r0 = (int64_t)c * N;
  const int n = (int)min((int64_t)N, rows - r0);
  const int t = threadIdx.x;
  const int pos0 = t * E;
  int v[E];
#pragma unroll
  for (int i = 0; i < E; ++i)
    v[i] = pos0 + i < n ? fkey(X[(r0 + pos0 + i) * ld + f]) : INT_MAX;
  for (int k = 2; k <= N; k <<= 1) {
    for (int j = k >> 1; j >= E; j >>= 1) {
      const int d = j / E;   // partner thread t ^ d, same slot
#pragma unroll
      for (int i = 0; i < E; ++i) sk[i * kSortThreads + t] = v[i];
      __syncthreads();
      const bool low = (t & d) == 0;
#pragma unroll
      for (int i = 0; i < E; ++i) {
        const int o = sk[i * kSortThreads + (t ^ d)];
        const bool up = ((pos0 + i) & k) == 0;
        v[i] = low == up ? min(v[i], o) : max(v[i], o);
      }
      __syncthreads();
    }
    register_stages<E, E / 2>(v, pos0, k);
  }
  int* out = keys + ((int64_t)f * chunks + c) * N;
#pragma unroll
  for (int i = 0; i < E; ++i) out[pos0 + i] = v[i];
}

// Group of bin bi (wave-uniform): the g with group_bins[g] <= bi < group_bins[g+1].
__device__ __forceinline__ int group_of_bin(const int32_t* __restrict__ group_bins, int G,
                                            int64_t bi) {
  int lo = 0, hi = G;   // group_bins[lo] <= bi < group_bins[hi]
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (group_bins[mid] <= bi) lo = mid;
    else hi = mid;
  }
  return lo;
}

// Lane view of one bin: every lane's element, the lane of its path's root,
// the path's length and zero-fraction count.
template <typename T>
struct BinLanes {
  int e0, len;
  int feat;
  bool root;
  uint64_t roots;
  int rl;     // lane of this lane's root
  int size;   // elements of this lane's path, root included
  int n0;     // zero-fraction elements of this lane's path
};

template <typename T>
__device__ __forceinline__ BinLanes<T> bin_lanes(const DevModel<T>& d, int64_t bi, int lane) {
  BinLanes<T> b;
  b.e0 = d.bin_start[bi];
  b.len = d.bin_start[bi + 1] - b.e0;
  b.feat = lane < b.len ? d.feat[b.e0 + lane] : 0;
  b.root = lane < b.len && b.feat < 0;
  b.roots = __ballot(b.root);
  const uint64_t upto = b.roots & ((2ull << lane) - 1ull);
  b.rl = upto ? 63 - __clzll((long long)upto) : lane;
  int size = 0;
  if (b.root) {
    const uint64_t above = b.roots & ~((2ull << lane) - 1ull);
    size = (above ? __builtin_ctzll(above) : b.len) - lane;
  }
  b.size = __shfl(size, b.rl);
  b.n0 = __shfl(b.root ? -1 - b.feat : 0, b.rl);
  return b;
}

// Partial counter of a workgroup of mark_paths / copy_paths (the same grid).
__device__ __forceinline__ int part_of_block() { return (int)(blockIdx.x % kParts); }

template <typename T>
__global__ __launch_bounds__(64 * kMarkWaves) void mark_paths(DevModel<T> d, int64_t num_bins,
                                                              const int* __restrict__ keys,
                                                              int64_t rows, int chunk, int chunks,
                                                              int* __restrict__ counts,
                                                              int* __restrict__ ranks) {
  const int lane = threadIdx.x & 63;
  const int64_t bi = (int64_t)blockIdx.x * kMarkWaves + (threadIdx.x >> 6);
  if (bi >= num_bins) return;   // the whole wave
  const BinLanes<T> b = bin_lanes(d, bi, lane);
  // a zero-fraction element: does any row's key lie in [klo, klo + span)?
  const int j = lane - b.rl - 1;
  bool miss = false;
  if (lane < b.len && !b.root && j < b.n0) {
    const int klo = fkey(d.lower[b.e0 + lane]);
    const unsigned span = key_span(klo, fkey(d.upper[b.e0 + lane]));
    bool hit = false;
    if (span != 0u) {
      const int khi = (int)((unsigned)klo + span);
      for (int c = 0; c < chunks && !hit; ++c) {
        const int n = (int)min((int64_t)chunk, rows - (int64_t)c * chunk);
        const int* s = keys + ((int64_t)b.feat * chunks + c) * chunk;
        int lo = 0, hi = n;   // the first key >= klo
        while (lo < hi) {
          const int mid = (lo + hi) >> 1;
          if (s[mid] < klo) lo = mid + 1;
          else hi = mid;
        }
        hit = lo < n && s[lo] < khi;
      }
    }
    miss = !hit;
  }
  const uint64_t misses = __ballot(miss);
  bool keep = false;
  if (b.root) {
    const uint64_t mine = (b.size >= 64 - lane ? ~0ull : ((1ull << (lane + b.size)) - 1ull)) &
                          ~((2ull << lane) - 1ull);
    keep = (misses & mine) == 0;
  }
  // ranks among the kept paths of this group and length: one atomic add per
  // length present in the wave
  const int g = group_of_bin(d.group_bins, d.G, bi);
  int* cnt = counts + (int64_t)g * kSizes * kParts;
  const int part = part_of_block();
  int rank = -1;
  for (uint64_t pend = __ballot(keep); pend != 0;) {
    const int first = __builtin_ctzll(pend);
    const int s0 = __shfl(b.size, first);
    const uint64_t same = __ballot(keep && b.size == s0);
    int base = 0;
    if (lane == first) base = atomicAdd(cnt + s0 * kParts + part, __popcll(same));
    base = __shfl(base, first);
    if (keep && b.size == s0) rank = base + __popcll(same & ((1ull << lane) - 1ull));
    pend &= ~same;
  }
  if (b.root) ranks[b.e0 + lane] = rank;
}

// Class q of the order group, length descending: group q / 64, length
// 64 - q % 64; its index in the [G][kSizes] arrays.
__device__ __forceinline__ int class_index(int q) {
  return (q / kMaxPathLen) * kSizes + (kMaxPathLen - q % kMaxPathLen);
}

// One workgroup: per (group, length) class, the kept paths' total and each
// partial counter's first rank; element and bin bases of the classes in the
// order group, length descending (a block-wide scan); every bin's start.
// counts[g][s][p] ends as the element offset of rank 0 of partial counter p.
constexpr int kPlanThreads = 1024;

template <typename T>
__global__ __launch_bounds__(kPlanThreads) void plan_pruned(int G, int* __restrict__ counts,
                                                            int* __restrict__ totals,
                                                            int32_t* __restrict__ bin_start,
                                                            int32_t* __restrict__ group_bins,
                                                            const T* __restrict__ bias_in,
                                                            T* __restrict__ bias_out) {
  __shared__ int se[kPlanThreads], sb[kPlanThreads];
  const int tid = threadIdx.x;
  const int Q = G * kMaxPathLen;
  for (int q = tid; q < Q; q += kPlanThreads) {
    int* p = counts + (int64_t)class_index(q) * kParts;
    int run = 0;
    for (int i = 0; i < kParts; ++i) {
      const int n = p[i];
      p[i] = run;
      run += n;
    }
    totals[2 * class_index(q)] = run;
  }
  for (int g = tid; g < G; g += kPlanThreads) bias_out[g] = bias_in[g];
  // exclusive scan of (elements, bins) over the classes, 1024 at a time
  int carry_e = 0, carry_b = 0;
  for (int q0 = 0; q0 < Q; q0 += kPlanThreads) {
    const int q = q0 + tid;
    int e = 0, b = 0;
    if (q < Q) {
      const int s = kMaxPathLen - q % kMaxPathLen;
      const int n = totals[2 * class_index(q)];   // written by this thread above
      const int per = kMaxPathLen / s;
      e = n * s;
      b = (n + per - 1) / per;
    }
    se[tid] = e;
    sb[tid] = b;
    __syncthreads();
    for (int off = 1; off < kPlanThreads; off <<= 1) {
      const int xe = tid >= off ? se[tid - off] : 0;
      const int xb = tid >= off ? sb[tid - off] : 0;
      __syncthreads();
      se[tid] += xe;
      sb[tid] += xb;
      __syncthreads();
    }
    if (q < Q) {
      totals[2 * class_index(q)] = carry_e + se[tid] - e;       // element base
      totals[2 * class_index(q) + 1] = carry_b + sb[tid] - b;   // bin base
    }
    carry_e += se[kPlanThreads - 1];
    carry_b += sb[kPlanThreads - 1];
    __syncthreads();
  }
  const int nb = carry_b;
  for (int g = tid; g < G; g += kPlanThreads)
    group_bins[g] = totals[2 * class_index(g * kMaxPathLen) + 1];
  if (tid == 0) {
    group_bins[G] = nb;
    bin_start[nb] = carry_e;
  }
  __syncthreads();   // the bases written above, for every thread
  for (int q = tid; q < Q; q += kPlanThreads) {
    const int c = class_index(q);
    const int s = kMaxPathLen - q % kMaxPathLen;
    const int el = totals[2 * c];
    int* p = counts + (int64_t)c * kParts;
    for (int i = 0; i < kParts; ++i) p[i] = el + p[i] * s;
  }
  // every bin's start: the last class whose bin base is <= the bin (classes
  // without bins share their successor's base and come before it)
  for (int bi = tid; bi < nb; bi += kPlanThreads) {
    int lo = 0, hi = Q;
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (totals[2 * class_index(mid) + 1] <= bi) lo = mid;
      else hi = mid;
    }
    const int c = class_index(lo);
    const int s = kMaxPathLen - lo % kMaxPathLen;
    bin_start[bi] = totals[2 * c] + (bi - totals[2 * c + 1]) * (kMaxPathLen / s) * s;
  }
}

template <typename T>
__global__ __launch_bounds__(64 * kMarkWaves) void copy_paths(DevModel<T> d, int64_t num_bins,
                                                              const int* __restrict__ counts,
                                                              const int* __restrict__ ranks,
                                                              int32_t* __restrict__ feat,
                                                              float* __restrict__ lower,
                                                              float* __restrict__ upper,
                                                              T* __restrict__ zero) {
  const int lane = threadIdx.x & 63;
  const int64_t bi = (int64_t)blockIdx.x * kMarkWaves + (threadIdx.x >> 6);
  if (bi >= num_bins) return;
  const BinLanes<T> b = bin_lanes(d, bi, lane);
  const int rank = __shfl(b.root ? ranks[b.e0 + lane] : -1, b.rl);
  if (lane >= b.len || rank < 0) return;
  const int g = group_of_bin(d.group_bins, d.G, bi);
  const int base = counts[((int64_t)g * kSizes + b.size) * kParts + part_of_block()];
  const int64_t dst = (int64_t)base + (int64_t)rank * b.size + (lane - b.rl);
  const int64_t src = b.e0 + lane;
  feat[dst] = b.feat;
  lower[dst] = d.lower[src];
  upper[dst] = d.upper[src];
  zero[dst] = d.zero[src];
}

template <typename T>
gts_status run_prune(const gts_model* m, const void* d_model, const float* X, int64_t rows,
                     int64_t ld, char* ws, const PruneLayout& L, hipStream_t stream) {
  const DevModel<T> d = dev_model<T>(m, d_model);
  const int M = m->num_features, G = m->num_groups;
  int* keys = reinterpret_cast<int*>(ws + L.keys);
  int* counts = reinterpret_cast<int*>(ws + L.counts);
  int* totals = reinterpret_cast<int*>(ws + L.totals);
  int* ranks = reinterpret_cast<int*>(ws + L.ranks);
  char* blob = ws + L.blob;
  const size_t lds = (size_t)L.chunk * sizeof(int);
  const int E = (int)(L.chunk / kSortThreads);
  const void* sorter = E == 1   ? reinterpret_cast<const void*>(sort_keys<1>)
                       : E == 2 ? reinterpret_cast<const void*>(sort_keys<2>)
                       : E == 4 ? reinterpret_cast<const void*>(sort_keys<4>)
                       : E == 8 ? reinterpret_cast<const void*>(sort_keys<8>)
                                : reinterpret_cast<const void*>(sort_keys<16>);
  if (hipFuncSetAttribute(sorter, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) !=
      hipSuccess) {
    (void)hipGetLastError();
    return fail(GTS_EDEVICE, "cannot set the LDS size of the key sort to %zu bytes", lds);
  }
  const dim3 sgrid((unsigned)(M * L.chunks)), sblock(kSortThreads);
  const int nch = (int)L.chunks;
  switch (E) {
    case 1: hipLaunchKernelGGL(sort_keys<1>, sgrid, sblock, lds, stream, X, rows, ld, M, nch, keys); break;
    case 2: hipLaunchKernelGGL(sort_keys<2>, sgrid, sblock, lds, stream, X, rows, ld, M, nch, keys); break;
    case 4: hipLaunchKernelGGL(sort_keys<4>, sgrid, sblock, lds, stream, X, rows, ld, M, nch, keys); break;
    case 8: hipLaunchKernelGGL(sort_keys<8>, sgrid, sblock, lds, stream, X, rows, ld, M, nch, keys); break;
    default: hipLaunchKernelGGL(sort_keys<16>, sgrid, sblock, lds, stream, X, rows, ld, M, nch, keys); break;
  }
  const int64_t ncount = (int64_t)G * kSizes * kParts;
  hipLaunchKernelGGL(fill_zero<int>, dim3((unsigned)std::min<int64_t>((ncount + 255) / 256, 4096)),
                     dim3(256), 0, stream, counts, ncount);
  const int64_t K = m->num_bins;
  const int64_t blocks = (K + kMarkWaves - 1) / kMarkWaves;
  if (blocks > 0x7fffffffLL) return fail(GTS_EINVAL, "too many bins for one launch");
  if (blocks > 0)
    hipLaunchKernelGGL(mark_paths<T>, dim3((unsigned)blocks), dim3(64 * kMarkWaves), 0, stream, d,
                       K, keys, rows, (int)L.chunk, (int)L.chunks, counts, ranks);
  hipLaunchKernelGGL(plan_pruned<T>, dim3(1), dim3(kPlanThreads), 0, stream, G, counts, totals,
                     reinterpret_cast<int32_t*>(blob + L.off[kBinStart]),
                     reinterpret_cast<int32_t*>(blob + L.off[kGroupBins]), d.bias,
                     reinterpret_cast<T*>(blob + L.off[kBias]));
  if (blocks > 0)
    hipLaunchKernelGGL(copy_paths<T>, dim3((unsigned)blocks), dim3(64 * kMarkWaves), 0, stream, d,
                       K, counts, ranks, reinterpret_cast<int32_t*>(blob + L.off[kFeat]),
                       reinterpret_cast<float*>(blob + L.off[kLower]),
                       reinterpret_cast<float*>(blob + L.off[kUpper]),
                       reinterpret_cast<T*>(blob + L.off[kZero]));
  const hipError_t err = hipGetLastError();
  if (err != hipSuccess) return fail(GTS_EDEVICE, "prune launch failed: %s", hipGetErrorString(err));
  return GTS_OK;
}

}  // namespace
}  // namespace gts

extern "C" gts_status gts_prune_workspace_bytes(const gts_model* model, int64_t rows,
                                                int64_t* bytes) {
  using namespace gts;
  clear_error();
  if (bytes == nullptr) return fail(GTS_EINVAL, "bytes must not be NULL");
  gts_status st = check_model(model);
  if (st != GTS_OK) return st;
  if (rows < 0) return fail(GTS_EINVAL, "rows must be >= 0");
  *bytes = prune_layout(model, rows, lds_per_block()).bytes;
  return GTS_OK;
}

extern "C" gts_status gts_prune_model(const gts_model* model, const void* d_model,
                                      const float* d_X, int64_t rows, int64_t ld_x,
                                      void* d_workspace, int64_t workspace_bytes,
                                      gts_model* pruned, void** d_pruned, void* stream) {
  using namespace gts;
  clear_error();
  gts_status st = check_model(model);
  if (st != GTS_OK) return st;
  if (model->flags & GTS_MODEL_PRUNED)
    return fail(GTS_EINVAL, "the model is already pruned (its counts are capacities)");
  if (pruned == nullptr || d_pruned == nullptr)
    return fail(GTS_EINVAL, "pruned and d_pruned must not be NULL");
  if (rows < 0) return fail(GTS_EINVAL, "rows must be >= 0");
  if (d_model == nullptr || d_workspace == nullptr || (rows > 0 && d_X == nullptr))
    return fail(GTS_EINVAL, "device pointers must not be NULL");
  if (rows > 0 && ld_x < model->num_features) return fail(GTS_EINVAL, "ld_x < num_features");
  if ((reinterpret_cast<uintptr_t>(d_workspace) & (uintptr_t)(kBlobAlign - 1)) != 0)
    return fail(GTS_EINVAL, "d_workspace must be aligned to %lld bytes", (long long)kBlobAlign);
  if (model->num_elements >= INT32_MAX || model->num_paths >= INT32_MAX)
    return fail(GTS_EINVAL, "model too large for 32-bit device indices");
  const PruneLayout L = prune_layout(model, rows, lds_per_block());
  if (workspace_bytes < L.bytes)
    return fail(GTS_EBUFSIZE, "workspace_bytes %lld < %lld", (long long)workspace_bytes,
                (long long)L.bytes);
  // the pruned model: the same arrays, in the workspace, with capacities of
  // the original's sizes; its bins hold one path length each
  gts_model pm = *model;
  for (int a = 0; a < kBlobArrays; ++a) pm.off[a] = L.off[a];
  pm.bytes = L.blob_bytes;
  pm.flags |= GTS_MODEL_SORTED_BINS | GTS_MODEL_PRUNED;
  char* ws = static_cast<char*>(d_workspace);
  if (rows > 0) {
    hipStream_t s = static_cast<hipStream_t>(stream);
    st = model->dtype == GTS_F64 ? run_prune<double>(model, d_model, d_X, rows, ld_x, ws, L, s)
                                 : run_prune<float>(model, d_model, d_X, rows, ld_x, ws, L, s);
    if (st != GTS_OK) return st;
  }
  *pruned = pm;
  *d_pruned = ws + L.blob;
  return GTS_OK;
}
