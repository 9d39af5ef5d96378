// Host half of libgts: argument checking, path extraction with duplicate
// merging (Sections 3.1-3.2), bin packing (Section 3.3) and the device
// layout.  Compiled without floating-point contraction so that the extracted
// zero fractions and the bias are reproducible bit for bit.
#include <algorithm>
#include <atomic>
#include <condition_variable>
#include <mutex>
#include <pthread.h>
#include <sched.h>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <functional>
#include <limits>
#include <memory>
#include <new>
#include <thread>
#include <type_traits>
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

// ---------------------------------------------------------------------------
// path extraction
// ---------------------------------------------------------------------------

// One split on the way from the root to a leaf.
struct Split {
  int32_t feature;
  float lower, upper;
  double zero_fraction;
};

// A merged element as an fp32 blob stores it: the zero fraction rounded to
// float (16 bytes instead of 24).
struct SplitF {
  int32_t feature;
  float lower, upper;
  float zero_fraction;
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

// Priority of a parallel region: the ticket of the host call it belongs to.
// A preparation takes a ticket when it starts (TicketScope); a region of a
// thread without one takes its own when it opens.  Both come from one
// counter, so a smaller ticket is an earlier start.
std::atomic<uint64_t> g_tickets{0};
thread_local uint64_t t_ticket = 0;

struct TicketScope {
  uint64_t saved;
  TicketScope() : saved(t_ticket) { t_ticket = g_tickets.fetch_add(1) + 1; }
  ~TicketScope() { t_ticket = saved; }
};

// A small persistent pool of worker threads for the host passes (tree walks,
// blob writing).  run(n, body) calls body() on the caller and on up to n-1
// workers at once; body pulls its work from a shared counter, so it is
// correct with any number of participants.  Regions opened by different
// threads (several preparations in flight at once) share one crew: a free
// worker joins the open region with the smallest ticket that still wants
// workers, so the preparation that started first gets every free worker and
// is done soonest, and the others take what it leaves (its serial parts, the
// end of its regions).  A region's caller closes it to further workers when
// its own body() returns and then waits for the workers that joined.  The
// pool is never destroyed (its threads end with the process) and a forked
// child starts a fresh one.
//
// Workers that find nothing to join poll a version word, bumped whenever a
// region opens, for a while (first with a pause instruction, then yielding
// the core) before they block on the condition variable, so back-to-back
// regions -- a model preparation runs several, a few hundred microseconds
// apart -- start without a wake-up through the kernel; the caller polls the
// count of joined workers the same way.
class Pool {
 public:
  static Pool& get() {
    static std::once_flag once;
    std::call_once(once, [] { pthread_atfork(nullptr, nullptr, [] { instance() = nullptr; }); });
    std::lock_guard<std::mutex> lock(create_mu());
    if (instance() == nullptr) instance() = new Pool();
    return *instance();
  }

  template <typename Body>
  void run(int n, Body&& body) {
    if (n <= 1) {
      body();
      return;
    }
    std::function<void()> fn(std::ref(body));
    Region r;
    r.job = &fn;
    r.want = std::min(n - 1, kMaxWorkers);
    r.ticket = t_ticket != 0 ? t_ticket : g_tickets.fetch_add(1) + 1;
    {
      std::lock_guard<std::mutex> lock(grow_mu_);
      while (workers_.load(std::memory_order_relaxed) < r.want) {
        std::thread([this] { loop(); }).detach();
        workers_.fetch_add(1, std::memory_order_relaxed);
      }
    }
    {
      SpinGuard g(list_);
      auto at = open_.begin();
      while (at != open_.end() && (*at)->ticket <= r.ticket) ++at;
      open_.insert(at, &r);
      version_.fetch_add(1, std::memory_order_release);
    }
    {
      // a worker about to sleep checks the version under sleep_mu_, so it
      // either sees the new one or is waiting when this notifies
      std::lock_guard<std::mutex> lock(sleep_mu_);
      if (sleepers_ > 0) cv_.notify_all();
    }
    // the region leaves the list, and every worker that joined it has left
    // it, before it goes out of scope, also when body() throws
    struct Close {
      Pool& p;
      Region& r;
      ~Close() {
        {
          SpinGuard g(p.list_);
          p.open_.erase(std::find(p.open_.begin(), p.open_.end(), &r));
        }
        // no worker joins a closed region; wait for those inside it
        for (int i = 0; r.active.load(std::memory_order_acquire) != 0; ++i) relax(i);
      }
    } close{*this, r};
    body();
  }

 private:
  static constexpr int kMaxWorkers = 63;
  static constexpr int kPauseRounds = 2048;     // ~ tens of microseconds
  static constexpr int kYieldRounds = 4096;     // then yield the core, ~ a millisecond

  struct Region {
    const std::function<void()>* job = nullptr;
    uint64_t ticket = 0;
    int want = 0;                   // workers that may still join (under list_)
    std::atomic<int> active{0};     // workers that joined and have not left
  };

  // The region list's lock: held for a few list operations at a time, by
  // callers opening or closing a region and by workers joining one, so a
  // waiter spins instead of sleeping in the kernel.
  struct SpinGuard {
    std::atomic_flag& f;
    explicit SpinGuard(std::atomic_flag& flag) : f(flag) {
      for (int i = 0; f.test_and_set(std::memory_order_acquire); ++i) relax(i);
    }
    ~SpinGuard() { f.clear(std::memory_order_release); }
  };

  static void relax(int i) {
#if defined(__x86_64__) || defined(__i386__)
    if (i < kPauseRounds) {
      __builtin_ia32_pause();
      return;
    }
#endif
    std::this_thread::yield();
  }

  static Pool*& instance() {
    static Pool* p = nullptr;
    return p;
  }
  static std::mutex& create_mu() {
    static std::mutex m;
    return m;
  }

  void loop() {
    for (;;) {
      Region* r = nullptr;
      uint64_t seen;
      {
        SpinGuard g(list_);
        for (Region* x : open_)
          if (x->want > 0) {
            r = x;
            break;
          }
        if (r != nullptr) {
          r->want -= 1;
          r->active.fetch_add(1, std::memory_order_relaxed);
        }
        seen = version_.load(std::memory_order_relaxed);
      }
      if (r != nullptr) {
        // the region stays alive until its caller has seen active drop to 0
        (*r->job)();
        r->active.fetch_sub(1, std::memory_order_release);
        continue;
      }
      int i = 0;
      while (version_.load(std::memory_order_acquire) == seen && i < kPauseRounds + kYieldRounds)
        relax(i++);
      if (version_.load(std::memory_order_acquire) == seen) {
        std::unique_lock<std::mutex> lock(sleep_mu_);
        ++sleepers_;
        cv_.wait(lock, [&] { return version_.load(std::memory_order_acquire) != seen; });
        --sleepers_;
      }
    }
  }

  std::atomic_flag list_ = ATOMIC_FLAG_INIT;
  std::vector<Region*> open_;         // under list_, ascending ticket
  std::atomic<uint64_t> version_{0};  // bumped (under list_) when a region opens
  std::mutex grow_mu_;                // starting workers
  std::atomic<int> workers_{0};
  std::mutex sleep_mu_;
  std::condition_variable cv_;
  int sleepers_ = 0;                  // under sleep_mu_
};

// Per-thread state for walking trees depth first.  The merged elements of the
// path from the root to the current node are kept up to date on the way down
// and restored on the way up (Section 3.2): for every feature on the path,
// the intersection of its ranges and the product of its zero fractions taken
// in root-to-leaf order, and the set of features on the path (a bit mask for
// up to 64 features, else a list kept in ascending order).
struct Walker {
  // A node still to visit: its parent (-1 for the root) and the side it hangs
  // on, and the undo depth of the parent's path.
  struct Frame {
    int32_t node;
    int32_t from;    // parent * 2 + (1 if the right child), -1 at the root
    int32_t depth;
  };
  struct Undo {
    int32_t feature;
    float lower, upper;
    double zero_fraction;
  };
  std::vector<Frame> stack;
  std::vector<Undo> undo;
  std::vector<int32_t> count;   // [M] splits on the path, per feature
  std::vector<float> lower;     // [M]
  std::vector<float> upper;     // [M]
  std::vector<double> zf;       // [M]
  std::vector<int32_t> active;  // M > 64: features with count > 0, ascending
  uint64_t mask = 0;            // M <= 64: bit f set when count[f] > 0
  std::vector<unsigned char> seen;
  bool small = true;
  bool clean = false;

  void reset(int32_t M, int32_t n) {
    const float inf = std::numeric_limits<float>::infinity();
    small = M <= 64;
    if (!clean || (int32_t)count.size() != M) {
      count.assign((size_t)M, 0);
      lower.assign((size_t)M, -inf);
      upper.assign((size_t)M, inf);
      zf.assign((size_t)M, 1.0);
      active.clear();
      mask = 0;
    }
    if (stack.size() < (size_t)n + 1) stack.resize((size_t)n + 1);
    if (undo.size() < (size_t)n + 1) undo.resize((size_t)n + 1);
    clean = false;
  }

  size_t active_count() const { return small ? (size_t)__builtin_popcountll(mask) : active.size(); }

  // The current leaf's merged elements, in ascending feature order, into
  // dst[0..active_count()); returns the product of their zero fractions (a
  // left fold in that order).
  template <typename S>
  double emit(S* dst) const {
    using Z = decltype(S::zero_fraction);
    double prod = 1.0;
    if (small) {
      size_t i = 0;
      for (uint64_t m = mask; m; m &= m - 1, ++i) {
        const int32_t f = __builtin_ctzll(m);
        dst[i] = S{f, lower[(size_t)f], upper[(size_t)f], (Z)zf[(size_t)f]};
        prod = prod * zf[(size_t)f];
      }
    } else {
      for (size_t i = 0; i < active.size(); ++i) {
        const size_t f = (size_t)active[i];
        dst[i] = S{active[i], lower[f], upper[f], (Z)zf[f]};
        prod = prod * zf[f];
      }
    }
    return prod;
  }

  // Enter a split on feature f (range [lo, hi), cover ratio) at undo depth u.
  // Without VALUES only the set of features on the path is kept.
  template <bool VALUES>
  void push(int32_t u, int32_t f, float lo, float hi, double ratio) {
    const size_t i = (size_t)f;
    Undo& e = undo[(size_t)u];
    e.feature = f;
    if (VALUES) {
      const float l0 = lower[i], u0 = upper[i];
      e.lower = l0;
      e.upper = u0;
      e.zero_fraction = zf[i];
      lower[i] = lo > l0 ? lo : l0;
      upper[i] = hi < u0 ? hi : u0;
      zf[i] = zf[i] * ratio;
    }
    if (small) {
      // no branch on whether the feature is already on the path
      ++count[i];
      mask |= 1ull << f;
    } else if (count[i]++ == 0) {
      active.push_back(f);
      size_t k = active.size() - 1;
      for (; k > 0 && active[k - 1] > f; --k) active[k] = active[k - 1];
      active[k] = f;
    }
  }

  template <bool VALUES>
  void pop(int32_t u) {
    const Undo& e = undo[(size_t)u];
    const size_t i = (size_t)e.feature;
    if (VALUES) {
      lower[i] = e.lower;
      upper[i] = e.upper;
      zf[i] = e.zero_fraction;
    }
    if (small) {
      mask &= ~((uint64_t)(--count[i] == 0) << e.feature);
    } else if (--count[i] == 0) {
      size_t k = 0;
      while (active[k] != e.feature) ++k;
      for (; k + 1 < active.size(); ++k) active[k] = active[k + 1];
      active.pop_back();
    }
  }

  // Depth-first walk of tree t, left child (x < t) first, validating every
  // node it reaches (without CHECK, for a tree an earlier walk has
  // validated, no node is checked).  Calls leaf(node, m) with m merged
  // elements (with EMIT, emit() gives them; without EMIT only m is
  // computed).  The stack holds nodes still to visit, each with the undo
  // depth of its parent's path: a visit first unwinds the path to that depth,
  // then enters the split from the parent (range from the parent's threshold
  // and the side, zero fraction child cover / parent cover).
  template <bool EMIT, bool CHECK = true, typename LeafFn>
  gts_status walk(const gts_ensemble* e, int64_t t, LeafFn&& leaf) {
    const int64_t base = e->tree_node_offsets[t];
    const int32_t n = (int32_t)(e->tree_node_offsets[t + 1] - base);
    reset(e->num_features, n);
    if (CHECK) seen.assign((size_t)n, 0);
    const int32_t* const left = e->left + base;
    const int32_t* const right = e->right + base;
    const int32_t* const feature = e->feature + base;
    const float* const threshold = e->threshold + base;
    const double* const cover = e->cover + base;
    const double* const value = e->value + base;
    const int32_t M = e->num_features;
    const float inf = std::numeric_limits<float>::infinity();
    Frame* const st = stack.data();
    int32_t sp = 0;   // frames on the stack
    int32_t ud = 0;   // undo depth of the current path
    st[sp++] = Frame{0, -1, 0};
    gts_status status = GTS_OK;
    while (sp > 0) {
      const Frame fr = st[--sp];
      while (ud > fr.depth) pop<EMIT>(--ud);
      const int32_t node = fr.node;
      if (fr.from >= 0) {
        const int32_t parent = fr.from >> 1;
        const float th = threshold[parent];
        const bool is_right = fr.from & 1;
        push<EMIT>(ud++, feature[parent], is_right ? th : -inf, is_right ? inf : th,
                   EMIT ? cover_ratio(cover[node], cover[parent]) : 0.0);
      }
      const int32_t a = left[node], b = right[node];
      if (CHECK) {
        if (seen[(size_t)node]) {
          status = fail(GTS_EINVAL, "tree %lld: node %d reached twice (cycle or shared child)",
                        (long long)t, node);
          break;
        }
        seen[(size_t)node] = 1;
        const double r = cover[node];
        if (!(r >= 0.0) || !std::isfinite(r)) {
          status = fail(GTS_EINVAL, "tree %lld node %d: cover must be finite and >= 0",
                        (long long)t, node);
          break;
        }
      }
      if (a < 0 && b < 0) {
        if (CHECK && !std::isfinite(value[node])) {
          status = fail(GTS_EINVAL, "tree %lld leaf %d: value is not finite", (long long)t, node);
          break;
        }
        leaf(node, active_count());
        continue;
      }
      if (!CHECK) {
        st[sp++] = Frame{b, node * 2 + 1, ud};
        st[sp++] = Frame{a, node * 2, ud};
        continue;
      }
      if (a < 0 || b < 0 || a >= n || b >= n) {
        status = fail(GTS_EINVAL, "tree %lld node %d: child index out of range", (long long)t,
                      node);
        break;
      }
      const int32_t d = feature[node];
      if (d < 0 || d >= M) {
        status = fail(GTS_EINVAL, "tree %lld node %d: feature %d outside [0, %d)", (long long)t,
                      node, d, M);
        break;
      }
      if (std::isnan(threshold[node])) {
        status = fail(GTS_EINVAL, "tree %lld node %d: threshold is NaN", (long long)t, node);
        break;
      }
      // a node reached twice is refused at its second visit, so every node
      // is pushed at most twice and the stack holds at most n + 1 frames
      if (sp + 2 > (int32_t)stack.size()) {
        status = fail(GTS_EINVAL, "tree %lld node %d: node reached twice (cycle or shared child)",
                      (long long)t, node);
        break;
      }
      st[sp++] = Frame{b, node * 2 + 1, ud};
      st[sp++] = Frame{a, node * 2, ud};
    }
    while (ud > 0) pop<EMIT>(--ud);
    clean = true;
    return status;
  }

  // walk() without values for up to 64 features: each stack frame carries
  // the mask of the features on its path, so a leaf's merged element count
  // is a popcount (no per-feature state, no undo).  The same node checks,
  // messages and leaf order as walk().
  struct MaskFrame {
    int32_t node;
    int32_t depth;   // splits from the root
    uint64_t mask;
    uint64_t dirs;   // bit k set when the k-th split sends the path right
  };
  std::vector<MaskFrame> mstack;

  template <typename LeafFn>
  gts_status count_walk(const gts_ensemble* e, int64_t t, LeafFn&& leaf) {
    const int64_t base = e->tree_node_offsets[t];
    const int32_t n = (int32_t)(e->tree_node_offsets[t + 1] - base);
    if (mstack.size() < (size_t)n + 1) mstack.resize((size_t)n + 1);
    seen.assign((size_t)n, 0);
    const int32_t* const left = e->left + base;
    const int32_t* const right = e->right + base;
    const int32_t* const feature = e->feature + base;
    const float* const threshold = e->threshold + base;
    const double* const cover = e->cover + base;
    const double* const value = e->value + base;
    const int32_t M = e->num_features;
    MaskFrame* const st = mstack.data();
    int32_t sp = 0;
    st[sp++] = MaskFrame{0, 0, 0, 0};
    while (sp > 0) {
      const MaskFrame fr = st[--sp];
      const int32_t node = fr.node;
      if (seen[(size_t)node])
        return fail(GTS_EINVAL, "tree %lld: node %d reached twice (cycle or shared child)",
                    (long long)t, node);
      seen[(size_t)node] = 1;
      const double r = cover[node];
      if (!(r >= 0.0) || !std::isfinite(r))
        return fail(GTS_EINVAL, "tree %lld node %d: cover must be finite and >= 0",
                    (long long)t, node);
      const int32_t a = left[node], b = right[node];
      if (a < 0 && b < 0) {
        if (!std::isfinite(value[node]))
          return fail(GTS_EINVAL, "tree %lld leaf %d: value is not finite", (long long)t, node);
        leaf(node, (size_t)__builtin_popcountll(fr.mask), fr.dirs, fr.depth);
        continue;
      }
      if (a < 0 || b < 0 || a >= n || b >= n)
        return fail(GTS_EINVAL, "tree %lld node %d: child index out of range", (long long)t,
                    node);
      const int32_t d = feature[node];
      if (d < 0 || d >= M)
        return fail(GTS_EINVAL, "tree %lld node %d: feature %d outside [0, %d)", (long long)t,
                    node, d, M);
      if (std::isnan(threshold[node]))
        return fail(GTS_EINVAL, "tree %lld node %d: threshold is NaN", (long long)t, node);
      if (sp + 2 > (int32_t)mstack.size())
        return fail(GTS_EINVAL, "tree %lld node %d: node reached twice (cycle or shared child)",
                    (long long)t, node);
      const uint64_t m = fr.mask | 1ull << d;
      const uint64_t right = fr.depth < 64 ? 1ull << fr.depth : 0;
      st[sp++] = MaskFrame{b, fr.depth + 1, m, fr.dirs | right};
      st[sp++] = MaskFrame{a, fr.depth + 1, m, fr.dirs};
    }
    return GTS_OK;
  }
};

// The bias of each output group from the paths' terms v * prod(z): every
// tree sums its own paths' terms in path order, then each group sums its
// trees' sums in tree order.  (A fixed two-level order that a device
// reduction reproduces bit for bit with one thread per tree.)  tree_paths:
// [T+1] first path of every tree.  bias[g] is overwritten.
void sum_bias(const gts_ensemble* e, const int64_t* tree_paths, const double* term,
              double* bias) {
  for (int32_t g = 0; g < e->num_groups; ++g) bias[g] = 0.0;
  for (int64_t t = 0; t < e->num_trees; ++t) {
    double s = 0.0;
    for (int64_t p = tree_paths[t]; p < tree_paths[t + 1]; ++p) s = s + term[p];
    bias[e->tree_group[t]] = bias[e->tree_group[t]] + s;
  }
}

// Cores this process may run on (its affinity mask, which a container's CPU
// share narrows; hardware_concurrency() counts every online core).
int usable_cores() {
  static const int n = [] {
    cpu_set_t set;
    CPU_ZERO(&set);
    if (sched_getaffinity(0, sizeof(set), &set) == 0 && CPU_COUNT(&set) > 0)
      return (int)CPU_COUNT(&set);
    const unsigned hw = std::thread::hardware_concurrency();
    return hw == 0 ? 1 : (int)hw;
  }();
  return n;
}

// Threads for a host call: at most 16, at least ~1k nodes (or elements)
// each.  A small call (under 128 k nodes or elements) leaves two of the
// process's cores to the caller's own threads (the calling program, the HIP
// runtime) when it has 8 or more: with every core taken, a 0.3 ms
// preparation's slowest tenth measured 40 % above its median.  A large one
// takes every core: the deep model (646 k nodes) prepares in 4.5 ms on 16
// threads against 5.0 ms on 14.
//
// gts_set_host_threads caps this for the calls of one thread.  Several
// preparations in flight at once prepare more models per second than one at
// a time, because no single preparation uses 16 cores fully (its packing is
// serial); they share the pool, which gives every free worker to the one
// that started first.
thread_local int32_t t_thread_cap = 0;

int host_threads(int64_t work) {
  int64_t cores = usable_cores();
  if (t_thread_cap > 0) cores = std::min<int64_t>(cores, t_thread_cap);
  const int64_t hw = cores >= 8 && work < (int64_t(1) << 17) ? cores - 2 : cores;
  const int64_t by_work = (work + 1023) / 1024;
  return (int)std::max<int64_t>(1, std::min<int64_t>({hw, 16, by_work}));
}

// Runs fn(t, walker) for every tree on the pool (dynamic chunks of trees);
// returns the per-tree statuses.
template <typename Fn>
void for_each_tree(const gts_ensemble* e, std::vector<gts_status>& status, Fn&& fn) {
  const int64_t T = e->num_trees;
  status.assign((size_t)T, GTS_OK);
  std::atomic<int64_t> next{0};
  const int64_t chunk = std::max<int64_t>(1, std::min<int64_t>(8, T / 64));
  Pool::get().run(host_threads(e->num_nodes), [&]() {
    static thread_local Walker w;
    for (;;) {
      const int64_t a = next.fetch_add(chunk);
      if (a >= T) break;
      const int64_t b = std::min(T, a + chunk);
      for (int64_t t = a; t < b; ++t) status[(size_t)t] = fn(t, w);
    }
  });
}

}  // namespace
}  // namespace gts

using namespace gts;

extern "C" {

const char* gts_last_error(void) { return g_error; }

const char* gts_version(void) { return "gts 0.1 (gfx950)"; }

gts_status gts_set_host_threads(int32_t n) {
  clear_error();
  if (n < 0) return fail(GTS_EINVAL, "n must be >= 0");
  t_thread_cap = n;
  return GTS_OK;
}

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
    const int64_t T = ens->num_trees;
    // pass 1: elements and paths per tree
    std::vector<int64_t> tree_elems((size_t)T + 1, 0), tree_paths((size_t)T + 1, 0);
    std::vector<gts_status> status;
    for_each_tree(ens, status, [&](int64_t t, Walker& w) {
      int64_t ne = 0, np = 0;
      gts_status s = w.walk<false>(ens, t, [&](int32_t, size_t m) {
        ne += (int64_t)m + 1;
        ++np;
      });
      tree_elems[(size_t)t + 1] = ne;
      tree_paths[(size_t)t + 1] = np;
      return s;
    });
    for (int64_t t = 0; t < T; ++t) {
      if (status[(size_t)t] != GTS_OK) {
        // re-walk the first bad tree here so the message is this thread's
        Walker w;
        return w.walk<false>(ens, t, [](int32_t, size_t) {});
      }
    }
    for (int64_t t = 0; t < T; ++t) {
      tree_elems[(size_t)t + 1] += tree_elems[(size_t)t];
      tree_paths[(size_t)t + 1] += tree_paths[(size_t)t];
    }
    const int64_t n = tree_elems[(size_t)T], paths = tree_paths[(size_t)T];
    *num_elements = n;
    *num_paths = paths;
    if (bias)
      for (int32_t g = 0; g < ens->num_groups; ++g) bias[g] = 0.0;
    if (out == nullptr && bias == nullptr) return GTS_OK;
    if (out != nullptr && n > capacity)
      return fail(GTS_EBUFSIZE, "capacity %lld < %lld elements", (long long)capacity,
                  (long long)n);
    // pass 2: write the elements; keep each path's bias term v * prod(z)
    std::vector<double> term(bias ? (size_t)paths : 0);
    for_each_tree(ens, status, [&](int64_t t, Walker& w) {
      const int64_t base = ens->tree_node_offsets[t];
      const int32_t group = ens->tree_group[t];
      int64_t k = tree_elems[(size_t)t];
      int64_t p = tree_paths[(size_t)t];
      const float inf = std::numeric_limits<float>::infinity();
      static thread_local std::vector<Split> merged;
      if (merged.size() < (size_t)ens->num_features) merged.resize((size_t)ens->num_features);
      return w.walk<true>(ens, t, [&](int32_t leaf, size_t m) {
        const double v = ens->value[base + leaf];
        const double prod = w.emit(merged.data());
        if (bias) term[(size_t)p] = v * prod;
        if (out) {
          gts_path_element* el = out + k;
          el[0].path_idx = p;
          el[0].feature_idx = -1;
          el[0].group = group;
          el[0].lower = -inf;
          el[0].upper = inf;
          el[0].zero_fraction = 1.0;
          el[0].v = v;
          for (size_t i = 0; i < m; ++i) {
            const Split& s = merged[i];
            el[i + 1].path_idx = p;
            el[i + 1].feature_idx = s.feature;
            el[i + 1].group = group;
            el[i + 1].lower = s.lower;
            el[i + 1].upper = s.upper;
            el[i + 1].zero_fraction = s.zero_fraction;
            el[i + 1].v = v;
          }
        }
        k += (int64_t)m + 1;
        ++p;
      });
    });
    if (bias) sum_bias(ens, tree_paths.data(), term.data(), bias);
    return GTS_OK;
  } catch (const std::bad_alloc&) {
    return fail(GTS_ENOMEM, "host allocation failed");
  }
}

}  // extern "C"

namespace gts {
namespace {

// ---------------------------------------------------------------------------
// bin packing
// ---------------------------------------------------------------------------

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
  int64_t first = 0;
  for (int64_t i = 0; i < n; ++i) {
    const gts_path_element& e = el[i];
    if (e.feature_idx == -1) {
      if (i > 0)
        paths.push_back(PathRef{first, (int32_t)std::min<int64_t>(i - first, INT32_MAX), el[first].group});
      first = i;
      if (num_groups > 0 && (e.group < 0 || e.group >= num_groups))
        return fail(GTS_EINVAL, "element %lld: group %d outside [0, %d)", (long long)i,
                    e.group, num_groups);
      continue;
    }
    const gts_path_element& root = el[first];
    if (e.feature_idx < -1 || (num_features > 0 && e.feature_idx >= num_features))
      return fail(GTS_EINVAL, "element %lld: feature %d out of range", (long long)i,
                  e.feature_idx);
    if (e.path_idx != root.path_idx || e.group != root.group)
      return fail(GTS_EINVAL, "element %lld does not belong to the path started at %lld",
                  (long long)i, (long long)first);
  }
  paths.push_back(PathRef{first, (int32_t)std::min<int64_t>(n - first, INT32_MAX), el[first].group});
  for (const PathRef& p : paths)
    if (p.size > max_len)
      return fail(GTS_EPATHLEN, "path at element %lld has length %d > %d", (long long)p.first,
                  p.size, max_len);
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

// Processing order of Section 3.3: by group; then (BFD, FFD) non-increasing
// size; ties by position.  The sort key of a path is
//   rank of its group among the groups present * nsize + (cap - size),
// nsize = cap + 1 for BFD and FFD; for Next-Fit and one-path-per-bin the
// size part is dropped (nsize = 1).
inline bool size_decreasing(int32_t alg) { return alg == GTS_PACK_BFD || alg == GTS_PACK_FFD; }
inline int64_t keys_per_group(int32_t cap, int32_t alg) {
  return size_decreasing(alg) ? (int64_t)cap + 1 : 1;
}
inline int32_t sort_key(int32_t grank, int32_t size, int32_t cap, int32_t alg) {
  return size_decreasing(alg) ? grank * (cap + 1) + (cap - size) : grank;
}

// A run of placements k .. k+n-1 (all of size s) that went into bin b one
// after another: placement k+i sits at element offset w + i*s of the bin and
// is the bin's (slot + i)-th path.
struct Fill {
  int64_t k;
  int32_t b;
  int32_t n;
  int32_t w;
  int32_t slot;
  int32_t s;
};

// The outcome of packing: the fills in placement order.  Per bin: group,
// elements, paths.  The bins' element ranges, and the bins' path ranges for a
// list of placements by bin.  Per placement k (the k-th path in processing
// order, order[k]), when expanded from the fills: its bin, its element offset
// inside the bin and its rank among the bin's paths.
struct Packing {
  std::vector<int64_t> order;        // [P] paths in processing order
  std::vector<Fill> fills;
  std::vector<int64_t> bin_at;       // [P] per placement (expand())
  std::vector<uint8_t> within_at;    // [P] per placement: element offset inside the bin
  std::vector<uint8_t> slot_at;      // [P] per placement: rank among the bin's paths
  std::vector<int32_t> bin_used;     // [K] elements in the bin
  std::vector<int32_t> bin_paths;    // [K] paths in the bin
  std::vector<int32_t> bin_group;    // [K]
  std::vector<int64_t> bin_offsets;  // [K+1] element ranges
  std::vector<int64_t> bin_first;    // [K+1] path ranges
  std::vector<int64_t> dest;         // [P] per path: packed element offset (assign_bins)
  int64_t K = 0;
  bool sorted = true;                // every bin's sizes non-increasing in placement order

  // The per-placement arrays from the fills.
  void expand(int64_t P) {
    bin_at.resize((size_t)P);
    within_at.resize((size_t)P);
    slot_at.resize((size_t)P);
    for (const Fill& f : fills)
      for (int32_t i = 0; i < f.n; ++i) {
        bin_at[(size_t)(f.k + i)] = f.b;
        within_at[(size_t)(f.k + i)] = (uint8_t)(f.w + i * f.s);
        slot_at[(size_t)(f.k + i)] = (uint8_t)(f.slot + i);
      }
  }
};

// Runs the heuristic over the placements in processing order.  key_start
// [ng * nsize + 1]: first placement of every sort key.  The size of a
// placement is the one its key encodes for BFD and FFD, size_at[k] for the
// others.  group_of_rank[r]: the group id of rank r.  The loop reads no
// per-path array for BFD and FFD and records one fill per run of placements
// that goes into one bin.
void place_paths(const int64_t* key_start, int32_t ng, const int32_t* group_of_rank,
                 const int32_t* size_at, int64_t P, int32_t cap, int32_t alg, Packing& pk) {
  pk.fills.clear();
  pk.bin_used.clear();
  pk.bin_paths.clear();
  pk.bin_group.clear();
  pk.sorted = true;
  int64_t K = 0;
  auto open_bin = [&](int32_t g) {
    pk.bin_used.push_back(0);
    pk.bin_paths.push_back(0);
    pk.bin_group.push_back(g);
    return K++;
  };
  // placements k .. k+n-1 (size s) go into bin b from element offset w on
  auto put = [&](int64_t k, int64_t b, int32_t n, int32_t w, int32_t s) {
    int32_t& paths = pk.bin_paths[(size_t)b];
    pk.fills.push_back(Fill{k, (int32_t)b, n, w, paths, s});
    paths += n;
    pk.bin_used[(size_t)b] = w + n * s;
  };
  const int64_t nsize = keys_per_group(cap, alg);
  std::vector<int32_t> resid;
  static thread_local std::vector<BinHeap> by_resid;
  by_resid.resize((size_t)cap + 1);
  for (int32_t r = 0; r < ng; ++r) {
    const int32_t g = group_of_rank[r];
    const int64_t i = key_start[r * nsize], j = key_start[(r + 1) * nsize];
    if (alg == GTS_PACK_BFD) {
      // open bins by residual in [1, cap]: a min-heap of bin numbers each,
      // and bit (residual - 1) of `open` set when that heap is not empty
      for (BinHeap& h : by_resid) h.clear();
      uint64_t open = 0;
      // Items of one size come in a run.  Once an item has gone into bin b
      // (the smallest residual that fits, every other fitting residual being
      // at least as large), b's new residual, if it still fits, is strictly
      // the smallest: the next items of the run go into b until it no longer
      // fits.  So a bin takes residual / s items of the run at once, the
      // placements item-by-item Best-Fit-Decreasing makes.
      for (int64_t kk = 0; kk < nsize; ++kk) {
        const int32_t s = cap - (int32_t)kk;
        const int64_t k1 = key_start[r * nsize + kk + 1];
        for (int64_t k = key_start[r * nsize + kk]; k < k1;) {
          int64_t b;
          int32_t res;
          const uint64_t fit = s >= 1 ? open >> (s - 1) : open;
          if (fit != 0) {
            res = s + __builtin_ctzll(fit);
            b = heap_pop(by_resid[(size_t)res]);
            if (by_resid[(size_t)res].empty()) open &= ~(1ull << (res - 1));
          } else {
            b = open_bin(g);
            res = cap;
          }
          const int32_t n = (int32_t)std::min<int64_t>(res / s, k1 - k);
          put(k, b, n, cap - res, s);
          k += n;
          res -= n * s;
          if (res > 0) {
            heap_push(by_resid[(size_t)res], b);
            open |= 1ull << (res - 1);
          }
        }
      }
    } else if (alg == GTS_PACK_FFD) {
      const int64_t first_bin = K;
      FirstFitTree tree(j - i);
      resid.assign((size_t)(j - i), 0);
      // As for BFD, a run of equal-size items fills the chosen bin: every
      // bin left of it is too full for this size, so it stays the leftmost
      // fit while it fits.
      for (int64_t kk = 0; kk < nsize; ++kk) {
        const int32_t s = cap - (int32_t)kk;
        const int64_t k1 = key_start[r * nsize + kk + 1];
        for (int64_t k = key_start[r * nsize + kk]; k < k1;) {
          int64_t local = tree.leftmost_at_least(s);
          if (local < 0) {
            local = open_bin(g) - first_bin;
            resid[(size_t)local] = cap;
          }
          int32_t res = resid[(size_t)local];
          const int32_t n = (int32_t)std::min<int64_t>(res / s, k1 - k);
          put(k, first_bin + local, n, cap - res, s);
          k += n;
          res -= n * s;
          resid[(size_t)local] = res;
          tree.set(local, res);
        }
      }
    } else if (alg == GTS_PACK_NF) {
      const int64_t first_bin = K;
      int32_t res = 0, last = INT32_MAX;
      for (int64_t k = i; k < j; ++k) {
        const int32_t s = size_at[k];
        if (K == first_bin || res < s) {
          open_bin(g);
          res = cap;
          last = INT32_MAX;
        }
        if (s > last) pk.sorted = false;
        last = s;
        put(k, K - 1, 1, cap - res, s);
        res -= s;
      }
    } else {
      for (int64_t k = i; k < j; ++k) put(k, open_bin(g), 1, 0, size_at[k]);
    }
  }
  pk.K = K;
  pk.bin_offsets.resize((size_t)K + 1);
  pk.bin_first.resize((size_t)K + 1);
  pk.bin_offsets[0] = 0;
  pk.bin_first[0] = 0;
  for (int64_t b = 0; b < K; ++b) {
    pk.bin_offsets[(size_t)b + 1] = pk.bin_offsets[(size_t)b] + pk.bin_used[(size_t)b];
    pk.bin_first[(size_t)b + 1] = pk.bin_first[(size_t)b] + pk.bin_paths[(size_t)b];
  }
}

// Section 3.3 on paths given by size and group (path order = input order):
// the processing order by a counting sort over the keys above, the
// heuristic, and (with layout) every path's packed element offset.
void assign_bins(const int32_t* size, const int32_t* group, int64_t P, int32_t cap, int32_t alg,
                 Packing& pk, bool layout) {
  std::vector<int32_t> groups;
  groups.reserve(16);
  for (int64_t i = 0; i < P; ++i)
    if (groups.empty() || groups.back() != group[i]) groups.push_back(group[i]);
  std::sort(groups.begin(), groups.end());
  groups.erase(std::unique(groups.begin(), groups.end()), groups.end());
  const int64_t nkeys = (int64_t)groups.size() * keys_per_group(cap, alg);
  std::vector<int64_t> start((size_t)nkeys + 1, 0);
  std::vector<int32_t> key((size_t)P);
  for (int64_t i = 0; i < P; ++i) {
    const int32_t g =
        (int32_t)(std::lower_bound(groups.begin(), groups.end(), group[i]) - groups.begin());
    key[(size_t)i] = sort_key(g, size[i], cap, alg);
    ++start[(size_t)key[(size_t)i] + 1];
  }
  for (size_t k = 1; k < start.size(); ++k) start[k] += start[k - 1];
  std::vector<int64_t> pos(start.begin(), start.end() - 1);
  pk.order.resize((size_t)P);
  std::vector<int32_t> size_at((size_t)P);
  for (int64_t i = 0; i < P; ++i) {
    const int64_t k = pos[(size_t)key[(size_t)i]]++;
    pk.order[(size_t)k] = i;
    size_at[(size_t)k] = size[i];
  }
  place_paths(start.data(), (int32_t)groups.size(), groups.data(), size_at.data(), P, cap, alg,
              pk);
  pk.expand(P);
  if (!layout) return;
  pk.dest.resize((size_t)P);
  for (int64_t k = 0; k < P; ++k)
    pk.dest[(size_t)pk.order[(size_t)k]] =
        pk.bin_offsets[(size_t)pk.bin_at[(size_t)k]] + pk.within_at[(size_t)k];
}

// ---------------------------------------------------------------------------
// device layout
// ---------------------------------------------------------------------------

struct BlobPlan {
  gts_model m;
  int64_t sizes[kBlobArrays];
};

BlobPlan plan_blob(int64_t n, int64_t P, int64_t K, int32_t M, int32_t G, int32_t dtype,
                   int32_t maxlen) {
  BlobPlan bp;
  const size_t ts = dtype == GTS_F64 ? sizeof(double) : sizeof(float);
  bp.sizes[kFeat] = 4 * n;
  bp.sizes[kLower] = 4 * n;
  bp.sizes[kUpper] = 4 * n;
  bp.sizes[kZero] = (int64_t)ts * n;
  bp.sizes[kBinStart] = 4 * (K + 1);
  bp.sizes[kGroupBins] = 4 * ((int64_t)G + 1);
  bp.sizes[kBias] = (int64_t)ts * G;
  gts_model& m = bp.m;
  std::memset(&m, 0, sizeof(m));
  m.magic = kModelMagic;
  m.dtype = dtype;
  m.num_features = M;
  m.num_groups = G;
  m.num_elements = n;
  m.num_paths = P;
  m.num_bins = K;
  m.max_path_len = std::min<int32_t>(maxlen, kMaxPathLen + 1);
  int64_t cur = 0;
  for (int k = 0; k < kBlobArrays; ++k) {
    m.off[k] = cur;
    cur += (bp.sizes[k] + kBlobAlign - 1) / kBlobAlign * kBlobAlign;
  }
  m.bytes = cur > 0 ? cur : kBlobAlign;
  return bp;
}

// GTS_MODEL_SORTED_BINS if the paths of every bin, in their order in the
// bin, never grow in length; from packed elements (roots have feature -1)
// and bin offsets (unusable offsets give 0).
int32_t sorted_bins_flag(const gts_path_element* packed, int64_t n, const int64_t* bin_offsets,
                         int64_t K) {
  if (packed == nullptr || bin_offsets == nullptr) return 0;
  for (int64_t b = 0; b < K; ++b) {
    int64_t a = bin_offsets[b];
    const int64_t e = bin_offsets[b + 1];
    if (a < 0 || e > n || e < a) return 0;
    int64_t prev = INT64_MAX;
    while (a < e) {
      int64_t m = a + 1;
      while (m < e && packed[m].feature_idx != -1) ++m;
      if (m - a > prev) return 0;
      prev = m - a;
      a = m;
    }
  }
  return GTS_MODEL_SORTED_BINS;
}

// Zero the alignment padding after each array (the arrays themselves are
// written in full), so equal models give byte-identical blobs.
void zero_padding(const BlobPlan& bp, char* blob) {
  for (int k = 0; k < kBlobArrays; ++k) {
    const int64_t a = bp.m.off[k] + bp.sizes[k];
    const int64_t b = (k + 1 < kBlobArrays) ? bp.m.off[k + 1] : bp.m.bytes;
    if (b > a) std::memset(blob + a, 0, (size_t)(b - a));
  }
}

// The parts of the blob that depend only on the packing and the bias.
void write_bins_and_bias(const BlobPlan& bp, char* blob, const int64_t* bin_offsets,
                         const int32_t* bin_group, const double* bias) {
  const gts_model& m = bp.m;
  int32_t* bstart = reinterpret_cast<int32_t*>(blob + m.off[kBinStart]);
  int32_t* gbins = reinterpret_cast<int32_t*>(blob + m.off[kGroupBins]);
  for (int64_t b = 0; b <= m.num_bins; ++b) bstart[b] = (int32_t)bin_offsets[b];
  for (int64_t g = 0; g <= m.num_groups; ++g) gbins[g] = 0;
  for (int64_t b = 0; b < m.num_bins; ++b) gbins[bin_group[b] + 1] += 1;
  for (int64_t g = 0; g < m.num_groups; ++g) gbins[g + 1] += gbins[g];
  if (m.dtype == GTS_F64) {
    double* bb = reinterpret_cast<double*>(blob + m.off[kBias]);
    for (int64_t g = 0; g < m.num_groups; ++g) bb[g] = bias[g];
  } else {
    float* bb = reinterpret_cast<float*>(blob + m.off[kBias]);
    for (int64_t g = 0; g < m.num_groups; ++g) bb[g] = (float)bias[g];
  }
}

// One element of the blob: the root's zero-fraction slot holds v.
inline void put_element(const gts_model& m, char* blob, int64_t i, int32_t feat, float lo,
                        float hi, double z_or_v) {
  reinterpret_cast<int32_t*>(blob + m.off[kFeat])[i] = feat;
  reinterpret_cast<float*>(blob + m.off[kLower])[i] = lo;
  reinterpret_cast<float*>(blob + m.off[kUpper])[i] = hi;
  if (m.dtype == GTS_F64) reinterpret_cast<double*>(blob + m.off[kZero])[i] = z_or_v;
  else reinterpret_cast<float*>(blob + m.off[kZero])[i] = (float)z_or_v;
}

// Device order of a path's feature elements.
//
// Zero-fraction elements come first, in feature order, and the root's feature
// slot holds -1 - (their count).  A row outside the range of such an element
// meets the factor z + o t = 0 of the path's weight polynomial, so the
// (row, path) contributes nothing; the kernels test these elements first and
// skip a path that no row of their tile reaches.
//
// The other elements are rotated.  The kernels may run several paths of a
// bin side by side, one per group of lanes, stepping through their elements
// together; paths that share a feature (often the same tree's upper splits)
// would then update the same phi-tile entry in the same step, which the
// kernels' compare-and-swap accumulation resolves by retrying.  SHAP
// arithmetic does not depend on the element order, so each path's
// feature-sorted remaining elements are rotated: paths are taken in their
// order in the bin, and each gets the rotation (tried from t mod q' for the
// t-th path, q' the number of elements rotated) that puts the fewest of its
// features at a position where an earlier path of the bin already has the
// same feature.
//
// When every launch of the model runs one path per wave (rotate false), the
// order decides no collisions and the remaining elements keep their feature
// order.
//
// f, z: the path's q feature elements in ascending feature order (z in the
// blob's precision); used[f] has bit k set when an earlier path of the bin
// stores feature f at position k.  Writes order[k] = the source index stored
// at position k and returns the number of zero-fraction elements.
template <typename Z>
int32_t device_order(const int32_t* f, const Z* z, int32_t q, int32_t t_in_bin,
                     const uint64_t* used, bool rotate, int32_t* order) {
  int32_t n0 = 0;
  for (int32_t j = 0; j < q; ++j)
    if (z[j] == Z(0)) order[n0++] = j;
  int32_t rest[kMaxPathLen];
  int32_t nr = 0;
  for (int32_t j = 0; j < q; ++j)
    if (z[j] != Z(0)) rest[nr++] = j;
  int32_t best = 0;
  if (rotate && nr > 1) {
    // cost[rho]: collisions if rest element i goes to position
    // n0 + (i - rho) mod nr
    int32_t cost[kMaxPathLen];
    for (int32_t k = 0; k < nr; ++k) cost[k] = 0;
    const uint64_t in_q = q >= 64 ? ~0ull : (1ull << q) - 1;
    const uint64_t below = n0 >= 64 ? ~0ull : (1ull << n0) - 1;
    for (int32_t i = 0; i < nr; ++i) {
      uint64_t bits = used[(size_t)f[rest[i]]] & in_q & ~below;
      while (bits) {
        const int32_t kk = __builtin_ctzll(bits) - n0;
        bits &= bits - 1;
        ++cost[i >= kk ? i - kk : i - kk + nr];
      }
    }
    int32_t rho = t_in_bin % nr, best_cost = INT32_MAX;
    for (int32_t c = 0; c < nr; ++c) {
      if (cost[rho] < best_cost) {
        best_cost = cost[rho];
        best = rho;
        if (best_cost == 0) break;
      }
      if (++rho == nr) rho = 0;
    }
  }
  int32_t src = best;
  for (int32_t k = 0; k < nr; ++k, ++src) {
    if (src == nr) src = 0;
    order[n0 + k] = rest[src];
  }
  return n0;
}

// Applies device_order to the paths of one bin of a blob written in packed
// order (root first, features ascending), in place.
template <typename Z>
void rotate_bin(int32_t* feat, float* lo, float* hi, Z* zf, int64_t a0, int64_t a1, bool rotate,
                std::vector<uint64_t>& used, std::vector<int32_t>& touched) {
  Z zbuf[kMaxPathLen];
  float lbuf[kMaxPathLen], hbuf[kMaxPathLen];
  int32_t fbuf[kMaxPathLen], order[kMaxPathLen];
  int32_t t = 0;
  int64_t a = a0;
  while (a < a1) {
    int64_t e = a + 1;
    while (e < a1 && feat[e] >= 0) ++e;
    const int32_t q = (int32_t)(e - a - 1);
    const int32_t n0 = device_order(feat + a + 1, zf + a + 1, q, t, used.data(), rotate, order);
    for (int32_t k = 0; k < q; ++k) {
      const int64_t src = a + 1 + order[k];
      fbuf[k] = feat[src];
      lbuf[k] = lo[src];
      hbuf[k] = hi[src];
      zbuf[k] = zf[src];
    }
    feat[a] = -1 - n0;
    for (int32_t k = 0; k < q; ++k) {
      feat[a + 1 + k] = fbuf[k];
      lo[a + 1 + k] = lbuf[k];
      hi[a + 1 + k] = hbuf[k];
      zf[a + 1 + k] = zbuf[k];
      uint64_t& m = used[(size_t)fbuf[k]];
      if (m == 0) touched.push_back(fbuf[k]);
      m |= 1ull << k;
    }
    ++t;
    a = e;
  }
  for (int32_t f : touched) used[(size_t)f] = 0;
  touched.clear();
}

// Applies rotate_bin to every bin of a written blob, bins spread over the pool.
void rotate_bins(const gts_model& m, char* blob, const int64_t* bin_offsets) {
  int32_t* feat = reinterpret_cast<int32_t*>(blob + m.off[kFeat]);
  float* lo = reinterpret_cast<float*>(blob + m.off[kLower]);
  float* hi = reinterpret_cast<float*>(blob + m.off[kUpper]);
  const int64_t K = m.num_bins;
  const bool rotate = !one_path_per_wave(m.num_features, m.dtype);
  std::atomic<int64_t> next{0};
  const int nthreads = host_threads(m.num_elements);
  // about eight chunks a thread, at most 64 bins each
  const int64_t chunk = std::max<int64_t>(1, std::min<int64_t>(64, K / (8 * nthreads)));
  Pool::get().run(nthreads, [&]() {
    std::vector<uint64_t> used((size_t)m.num_features, 0);
    std::vector<int32_t> touched;
    for (;;) {
      const int64_t b0 = next.fetch_add(chunk);
      if (b0 >= K) break;
      const int64_t b1 = std::min(K, b0 + chunk);
      for (int64_t b = b0; b < b1; ++b) {
        if (m.dtype == GTS_F64)
          rotate_bin(feat, lo, hi, reinterpret_cast<double*>(blob + m.off[kZero]), bin_offsets[b],
                     bin_offsets[b + 1], rotate, used, touched);
        else
          rotate_bin(feat, lo, hi, reinterpret_cast<float*>(blob + m.off[kZero]), bin_offsets[b],
                     bin_offsets[b + 1], rotate, used, touched);
      }
    }
  });
}

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
    std::vector<int32_t> size((size_t)P), group((size_t)P);
    for (int64_t p = 0; p < P; ++p) {
      size[(size_t)p] = paths[(size_t)p].size;
      group[(size_t)p] = paths[(size_t)p].group;
    }
    Packing pk;
    const bool want = offsets_capacity > 0;
    assign_bins(size.data(), group.data(), P, bin_capacity, alg, pk, want);
    *num_bins = pk.K;
    if (!want) return GTS_OK;
    if (offsets_capacity < pk.K + 1)
      return fail(GTS_EBUFSIZE, "offsets_capacity %lld < num_bins + 1 = %lld",
                  (long long)offsets_capacity, (long long)(pk.K + 1));
    for (int64_t b = 0; b <= pk.K; ++b) bin_offsets[b] = pk.bin_offsets[(size_t)b];
    for (int64_t p = 0; p < P; ++p)
      std::memcpy(packed + pk.dest[(size_t)p], elems + paths[(size_t)p].first,
                  sizeof(gts_path_element) * (size_t)paths[(size_t)p].size);
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
  if (num_elements > 0 && packed == nullptr) return fail(GTS_EINVAL, "packed must not be NULL");
  if (blob_capacity < 0 || (blob_capacity > 0 && host_blob == nullptr))
    return fail(GTS_EINVAL, "bad host_blob / blob_capacity");
  try {
    // sizes: only counts are needed
    int64_t P = 0;
    int32_t maxlen = 0;
    {
      int64_t last = -1;
      for (int64_t i = 0; i < num_elements; ++i) {
        if (packed[i].feature_idx == -1) {
          if (last >= 0) maxlen = std::max<int32_t>(maxlen, (int32_t)std::min<int64_t>(i - last, INT32_MAX));
          last = i;
          ++P;
        }
      }
      if (last >= 0) maxlen = std::max<int32_t>(maxlen, (int32_t)std::min<int64_t>(num_elements - last, INT32_MAX));
    }
    BlobPlan bp = plan_blob(num_elements, P, num_bins, num_features, num_groups, dtype, maxlen);
    bp.m.flags = sorted_bins_flag(packed, num_elements, bin_offsets, num_bins);
    if (host_blob == nullptr) {
      *model = bp.m;
      return GTS_OK;
    }
    // full validation before anything is written
    std::vector<PathRef> paths;
    gts_status st = parse_paths(packed, num_elements, paths, kMaxPathLen, num_groups, num_features);
    if (st != GTS_OK) return st;
    if (bin_offsets[0] != 0 || bin_offsets[num_bins] != num_elements)
      return fail(GTS_EINVAL, "bin_offsets must run from 0 to num_elements");
    // every bin starts on a root element and holds whole paths of one group
    std::vector<int32_t> bin_group((size_t)num_bins);
    {
      size_t p = 0;
      for (int64_t b = 0; b < num_bins; ++b) {
        const int64_t a = bin_offsets[b], e = bin_offsets[b + 1];
        if (e < a || e - a > kMaxPathLen)
          return fail(GTS_EINVAL, "bin %lld spans %lld elements", (long long)b, (long long)(e - a));
        if (a == e) return fail(GTS_EINVAL, "bin %lld is empty", (long long)b);
        if (p >= paths.size() || paths[p].first != a)
          return fail(GTS_EINVAL, "bin %lld does not start on a path root", (long long)b);
        bin_group[(size_t)b] = paths[p].group;
        for (; p < paths.size() && paths[p].first < e; ++p) {
          if (paths[p].first + paths[p].size > e)
            return fail(GTS_EINVAL, "a path crosses the end of bin %lld", (long long)b);
          if (paths[p].group != bin_group[(size_t)b])
            return fail(GTS_EINVAL, "bin %lld mixes output groups", (long long)b);
        }
        if (b > 0 && bin_group[(size_t)b] < bin_group[(size_t)b - 1])
          return fail(GTS_EINVAL, "bins must be ordered by group");
      }
    }
    *model = bp.m;
    if (blob_capacity < bp.m.bytes)
      return fail(GTS_EBUFSIZE, "blob_capacity %lld < %lld bytes", (long long)blob_capacity,
                  (long long)bp.m.bytes);
    char* blob = static_cast<char*>(host_blob);
    zero_padding(bp, blob);
    for (int64_t i = 0; i < num_elements; ++i) {
      const gts_path_element& e = packed[i];
      put_element(bp.m, blob, i, e.feature_idx, e.lower, e.upper,
                  e.feature_idx == -1 ? e.v : e.zero_fraction);
    }
    rotate_bins(bp.m, blob, bin_offsets);
    write_bins_and_bias(bp, blob, bin_offsets, bin_group.data(), bias);
    return GTS_OK;
  } catch (const std::bad_alloc&) {
    return fail(GTS_ENOMEM, "host allocation failed");
  }
}

namespace gts {
namespace {

// One tree's paths from a single walk: merged feature elements of every path
// (concatenated, ascending feature order), with each path's length (root
// included) and leaf value, and the tree's part of the bias.
// (aligned to keep the vector headers of trees that different threads fill
// at the same time on different cache lines)
// A growable array of trivially copyable elements whose new slots are left
// uninitialised (std::vector::resize would zero them first: twice the
// writes).
template <typename T>
struct RawBuf {
  std::unique_ptr<T[]> data;
  size_t size = 0, cap = 0;
  T* grow(size_t n) {
    if (size + n > cap) {
      const size_t c = std::max(size + n, 2 * cap + 64);
      std::unique_ptr<T[]> d(new T[c]);
      if (size) std::memcpy(d.get(), data.get(), size * sizeof(T));
      data = std::move(d);
      cap = c;
    }
    T* p = data.get() + size;
    size += n;
    return p;
  }
};

struct alignas(128) TreeOut {
  RawBuf<Split> el;            // fp64 models
  RawBuf<SplitF> elf;          // fp32 models
  std::vector<int64_t> first;  // per path: its first element in el / elf
  std::vector<int32_t> size;
  std::vector<double> v;
  std::vector<uint64_t> dirs;  // per path, for a plan: bit k set when its k-th
                               // split from the root sends it right
  bool too_deep = false;       // a path of more than 64 splits (no plan)
  double term_sum = 0.0;       // the terms v * prod(z) summed in path order
  int32_t max_size = 0;
  int64_t elements = 0;        // sum of size
  void clear() {
    el.size = 0;
    elf.size = 0;
    first.clear();
    size.clear();
    v.clear();
    dirs.clear();
    too_deep = false;
    term_sum = 0.0;
    max_size = 0;
    elements = 0;
  }
};

// A path as the blob writer reads it: its feature-sorted merged elements (in
// its tree's buffer), leaf value and feature count, and, once placed, its
// element offset inside its bin.
struct PathSrc {
  const void* el;   // Split for fp64 models, SplitF for fp32
  double v;
  int32_t q;
  int32_t within;
};

// Working arrays of gts_prepare_model, kept per calling thread between calls
// so that repeated preparations reuse their memory.
struct PrepareScratch {
  std::vector<TreeOut> trees;
  std::vector<int64_t> tree_first, chunk_start, key_start;
  std::vector<int32_t> size_at, key, grank, group_of_rank;
  std::vector<PathSrc> src_at, src_by_bin;   // per placement; per bin slot
  std::vector<int32_t> kpos, d_at;           // per path: its placement; per placement: its offset
  Packing pk;
};

// Writes one path, the walker's current leaf, to its place in the blob (root
// at element offset d, then its elements in device_order without rotation);
// returns the product of the zero fractions as emit() does.  For up to 64
// features each element goes straight to its slot: its rank among the
// zero-fraction features of the path, or after them among the others, from
// masks, with no branch on the values.
template <typename Z>
double put_path(const gts_model& m, char* blob, const Walker& w, size_t q, double v, int64_t d) {
  int32_t* const feat = reinterpret_cast<int32_t*>(blob + m.off[kFeat]) + d;
  float* const lower = reinterpret_cast<float*>(blob + m.off[kLower]) + d;
  float* const upper = reinterpret_cast<float*>(blob + m.off[kUpper]) + d;
  Z* const zero = reinterpret_cast<Z*>(blob + m.off[kZero]) + d;
  if (w.small) {
    const uint64_t mask = w.mask;
    uint64_t zmask = 0;   // features whose zero fraction is 0 in the blob's precision
    for (uint64_t mm = mask; mm; mm &= mm - 1) {
      const int32_t f = __builtin_ctzll(mm);
      zmask |= (uint64_t)((Z)w.zf[(size_t)f] == Z(0)) << f;
    }
    const int32_t n0 = __builtin_popcountll(zmask);
    feat[0] = -1 - n0;
    lower[0] = -std::numeric_limits<float>::infinity();
    upper[0] = std::numeric_limits<float>::infinity();
    zero[0] = (Z)v;
    double prod = 1.0;
    int32_t iz = 1, ir = 1 + n0;
    for (uint64_t mm = mask; mm; mm &= mm - 1) {
      const int32_t f = __builtin_ctzll(mm);
      const int32_t isz = (int32_t)((zmask >> f) & 1ull);
      const int32_t k = isz ? iz : ir;
      iz += isz;
      ir += 1 - isz;
      const double z = w.zf[(size_t)f];
      feat[k] = f;
      lower[k] = w.lower[(size_t)f];
      upper[k] = w.upper[(size_t)f];
      zero[k] = (Z)z;
      prod = prod * z;
    }
    return prod;
  }
  using S = std::conditional_t<std::is_same_v<Z, float>, SplitF, Split>;
  S el[kMaxPathLen];
  const double prod = w.emit(el);
  int32_t fs[kMaxPathLen], order[kMaxPathLen];
  Z zs[kMaxPathLen];
  for (size_t j = 0; j < q; ++j) {
    fs[j] = el[j].feature;
    zs[j] = (Z)el[j].zero_fraction;
  }
  const int32_t n0 = device_order(fs, zs, (int32_t)q, 0, nullptr, false, order);
  feat[0] = -1 - n0;
  lower[0] = -std::numeric_limits<float>::infinity();
  upper[0] = std::numeric_limits<float>::infinity();
  zero[0] = (Z)v;
  for (size_t k = 0; k < q; ++k) {
    const S& e = el[order[k]];
    feat[k + 1] = e.feature;
    lower[k + 1] = e.lower;
    upper[k + 1] = e.upper;
    zero[k + 1] = zs[order[k]];
  }
  return prod;
}

// Writes the paths of bin b into the blob, in the device order of
// device_order (the choices rotate_bin makes, taken from the feature-sorted
// source).  src[bin_first[b] ..]: the paths of bin b in placement order;
// src has P entries, of which the writer prefetches a few ahead.
template <typename Z>
void write_bin(const gts_model& m, char* blob, const Packing& pk, const PathSrc* src, int64_t P,
               int64_t b, std::vector<uint64_t>& used, std::vector<int32_t>& touched) {
  constexpr int64_t kAhead = 4;
  const float inf = std::numeric_limits<float>::infinity();
  int32_t* const feat = reinterpret_cast<int32_t*>(blob + m.off[kFeat]);
  float* const lower = reinterpret_cast<float*>(blob + m.off[kLower]);
  float* const upper = reinterpret_cast<float*>(blob + m.off[kUpper]);
  Z* const zero = reinterpret_cast<Z*>(blob + m.off[kZero]);
  uint64_t* const u = used.data();
  int32_t fs[kMaxPathLen], order[kMaxPathLen];
  Z zs[kMaxPathLen];
  int32_t t_in_bin = 0;
  const int64_t base = pk.bin_offsets[(size_t)b];
  const bool rotate = !one_path_per_wave(m.num_features, m.dtype);
  for (int64_t i = pk.bin_first[(size_t)b]; i < pk.bin_first[(size_t)b + 1]; ++i, ++t_in_bin) {
    if (i + kAhead < P) {
      const char* ahead = reinterpret_cast<const char*>(src[i + kAhead].el);
      __builtin_prefetch(ahead);
      __builtin_prefetch(ahead + 64);
      __builtin_prefetch(ahead + 128);
    }
    const PathSrc& ps = src[i];
    using S = std::conditional_t<std::is_same_v<Z, float>, SplitF, Split>;
    const S* el = static_cast<const S*>(ps.el);
    const int32_t q = ps.q;
    const int64_t d = base + ps.within;
    for (int32_t jj = 0; jj < q; ++jj) {
      fs[jj] = el[jj].feature;
      zs[jj] = (Z)el[jj].zero_fraction;
    }
    const int32_t n0 = device_order(fs, zs, q, t_in_bin, u, rotate, order);
    feat[d] = -1 - n0;
    lower[d] = -inf;
    upper[d] = inf;
    zero[d] = (Z)ps.v;
    for (int32_t kk = 0; kk < q; ++kk) {
      const S& e = el[order[kk]];
      const int64_t o = d + 1 + kk;
      feat[o] = e.feature;
      lower[o] = e.lower;
      upper[o] = e.upper;
      zero[o] = zs[order[kk]];
      uint64_t& bits = u[e.feature];
      if (bits == 0) touched.push_back(e.feature);
      bits |= 1ull << kk;
    }
  }
  for (int32_t f : touched) used[(size_t)f] = 0;
  touched.clear();
}

}  // namespace
}  // namespace gts

namespace gts {
namespace {

// Where gts_plan_model's outputs go (absent for gts_prepare_model).
struct PlanOut {
  gts_plan* plan;
  char* host_plan;      // NULL: sizes only
  int64_t capacity;
};

gts_status prepare_model(const gts_ensemble* ens, int32_t bin_capacity, int32_t alg,
                         int32_t dtype, gts_model* model, void* host_blob,
                         int64_t blob_capacity, double* bias, const PlanOut* po) {
  clear_error();
  const TicketScope ticket;   // this preparation's regions, before later ones
  if (model == nullptr) return fail(GTS_EINVAL, "model must not be NULL");
  if (bin_capacity < 1 || bin_capacity > kMaxPathLen)
    return fail(GTS_EINVAL, "bin_capacity %d outside [1, %d]", bin_capacity, kMaxPathLen);
  if (alg < GTS_PACK_BFD || alg > GTS_PACK_NONE)
    return fail(GTS_EINVAL, "unknown packing algorithm %d", alg);
  if (dtype != GTS_F32 && dtype != GTS_F64) return fail(GTS_EINVAL, "unknown dtype %d", dtype);
  if (blob_capacity < 0 || (blob_capacity > 0 && host_blob == nullptr))
    return fail(GTS_EINVAL, "bad host_blob / blob_capacity");
  gts_status st = validate_ensemble(ens);
  if (st != GTS_OK) return st;
  try {
    const int64_t T = ens->num_trees;
    const bool sizes_only = host_blob == nullptr && bias == nullptr;
    // When every launch of the model runs one path per wave, a path's order
    // in the blob does not depend on the other paths of its bin: the first
    // walk then only counts, and a second walk after the packing writes every
    // path straight to its place in the blob ("direct").  Otherwise one walk
    // keeps every path's merged elements (only their count for a size query)
    // per tree, and the bins are written from them.  The pool's workers write
    // into the calling thread's scratch.
    if (po != nullptr && !one_path_per_wave(ens->num_features, dtype))
      return fail(GTS_EINVAL,
                  "a plan needs a model whose every launch runs one path per wave "
                  "(M <= 17 in fp32, M <= 11 in fp64); M = %d", ens->num_features);
    const bool direct =
        (host_blob != nullptr && one_path_per_wave(ens->num_features, dtype)) || po != nullptr;
    const bool count_only = sizes_only || direct;
    static thread_local PrepareScratch tls;
    PrepareScratch& sc = tls;
    std::vector<TreeOut>& trees = sc.trees;
    if ((int64_t)trees.size() < T) trees.resize((size_t)T);
    std::vector<gts_status> status;
    for_each_tree(ens, status, [&](int64_t t, Walker& w) {
      TreeOut& out = trees[(size_t)t];
      out.clear();
      if (count_only) {
        auto count = [&](int32_t, size_t m, uint64_t dirs = 0, int32_t depth = 0) {
          out.size.push_back((int32_t)m + 1);
          out.max_size = std::max(out.max_size, (int32_t)m + 1);
          out.elements += (int64_t)m + 1;
          if (po != nullptr) {
            out.dirs.push_back(dirs);
            out.too_deep |= depth > 64;
          }
        };
        return ens->num_features <= 64 ? w.count_walk(ens, t, count) : w.walk<false>(ens, t, count);
      }
      const int64_t base = ens->tree_node_offsets[t];
      return w.walk<true>(ens, t, [&](int32_t leaf, size_t m) {
        const double v = ens->value[base + leaf];
        double prod;
        if (dtype == GTS_F64) {
          out.first.push_back((int64_t)out.el.size);
          prod = w.emit(out.el.grow(m));
        } else {
          out.first.push_back((int64_t)out.elf.size);
          prod = w.emit(out.elf.grow(m));
        }
        out.size.push_back((int32_t)m + 1);
        out.v.push_back(v);
        out.term_sum = out.term_sum + v * prod;
        out.max_size = std::max(out.max_size, (int32_t)m + 1);
        out.elements += (int64_t)m + 1;
      });
    });
    for (int64_t t = 0; t < T; ++t)
      if (status[(size_t)t] != GTS_OK) {
        Walker w;
        return w.walk<false>(ens, t, [](int32_t, size_t) {});
      }
    std::vector<int64_t>& tree_first = sc.tree_first;
    tree_first.assign((size_t)T + 1, 0);
    int64_t n = 0;
    int32_t maxlen = 0;
    for (int64_t t = 0; t < T; ++t) {
      const TreeOut& tr = trees[(size_t)t];
      tree_first[(size_t)t + 1] = tree_first[(size_t)t] + (int64_t)tr.size.size();
      n += tr.elements;
      maxlen = std::max(maxlen, tr.max_size);
    }
    const int64_t P = tree_first[(size_t)T];
    if (maxlen > bin_capacity)
      return fail(GTS_EPATHLEN, "a merged path has length %d > bin capacity %d", maxlen,
                  bin_capacity);
    if (n >= std::numeric_limits<int32_t>::max())
      return fail(GTS_EINVAL, "too many path elements for 32-bit device indices");

    // processing order (a counting sort on the keys of sort_key), over
    // chunks of consecutive trees on the pool: each chunk counts its keys,
    // then places its paths after those of every smaller key and of the
    // same key in earlier chunks -- the order of the serial sort
    std::vector<int32_t>& grank = sc.grank;
    std::vector<int32_t>& group_of_rank = sc.group_of_rank;
    grank.assign((size_t)ens->num_groups, -1);
    group_of_rank.clear();
    for (int64_t t = 0; t < T; ++t) grank[(size_t)ens->tree_group[t]] = 0;
    for (int32_t g = 0; g < ens->num_groups; ++g)
      if (grank[(size_t)g] == 0) {
        grank[(size_t)g] = (int32_t)group_of_rank.size();
        group_of_rank.push_back(g);
      }
    const int32_t ng = (int32_t)group_of_rank.size();
    const int64_t nkeys = (int64_t)ng * keys_per_group(bin_capacity, alg);
    const int nthreads = host_threads(n);
    const int64_t chunks = std::max<int64_t>(
        1, std::min<int64_t>({T, 4 * (int64_t)nthreads, P / std::max<int64_t>(1, 4 * nkeys)}));
    const bool need_size = !size_decreasing(alg);
    std::vector<int32_t>& key = sc.key;
    std::vector<int32_t>& size_at = sc.size_at;
    std::vector<int64_t>& start = sc.chunk_start;
    std::vector<int64_t>& key_start = sc.key_start;
    key.resize((size_t)P);
    if (need_size) size_at.resize((size_t)P);
    start.assign((size_t)(chunks * nkeys), 0);
    key_start.resize((size_t)nkeys + 1);
    auto chunk_trees = [&](int64_t c, int64_t& t0, int64_t& t1) {
      t0 = T * c / chunks;
      t1 = T * (c + 1) / chunks;
    };
    const int sort_threads = (int)std::min<int64_t>(nthreads, chunks);
    {
      std::atomic<int64_t> next{0};
      Pool::get().run(sort_threads, [&]() {
        for (int64_t c; (c = next.fetch_add(1)) < chunks;) {
          int64_t t0, t1;
          chunk_trees(c, t0, t1);
          int64_t* cnt = start.data() + c * nkeys;
          for (int64_t t = t0; t < t1; ++t) {
            const std::vector<int32_t>& sz = trees[(size_t)t].size;
            const int32_t r = grank[(size_t)ens->tree_group[t]];
            int64_t p = tree_first[(size_t)t];
            for (size_t k = 0; k < sz.size(); ++k, ++p) {
              const int32_t kk = sort_key(r, sz[k], bin_capacity, alg);
              key[(size_t)p] = kk;
              ++cnt[kk];
            }
          }
        }
      });
    }
    {
      int64_t run = 0;
      for (int64_t k = 0; k < nkeys; ++k) {
        key_start[(size_t)k] = run;
        for (int64_t c = 0; c < chunks; ++c) {
          int64_t& x = start[(size_t)(c * nkeys + k)];
          const int64_t cnt = x;
          x = run;
          run += cnt;
        }
      }
      key_start[(size_t)nkeys] = run;
    }
    Packing& pk = sc.pk;
    std::vector<PathSrc>& src_at = sc.src_at;
    std::vector<int32_t>& kpos = sc.kpos;
    if (direct) kpos.resize((size_t)P);
    else if (!sizes_only) src_at.resize((size_t)P);
    {
      std::atomic<int64_t> next{0};
      Pool::get().run(sort_threads, [&]() {
        for (int64_t c; (c = next.fetch_add(1)) < chunks;) {
          int64_t t0, t1;
          chunk_trees(c, t0, t1);
          int64_t* pos = start.data() + c * nkeys;
          for (int64_t t = t0; t < t1; ++t) {
            const TreeOut& tr = trees[(size_t)t];
            const std::vector<int32_t>& sz = tr.size;
            int64_t p = tree_first[(size_t)t];
            for (size_t j = 0; j < sz.size(); ++j, ++p) {
              const int64_t k = pos[key[(size_t)p]]++;
              if (direct)
                kpos[(size_t)p] = (int32_t)k;
              else if (!sizes_only)
                src_at[(size_t)k] =
                    PathSrc{dtype == GTS_F64 ? (const void*)(tr.el.data.get() + tr.first[j])
                                             : (const void*)(tr.elf.data.get() + tr.first[j]),
                            tr.v[j], sz[j] - 1, 0};
              if (need_size) size_at[(size_t)k] = sz[j];
            }
          }
        }
      });
    }
    place_paths(key_start.data(), ng, group_of_rank.data(), need_size ? size_at.data() : nullptr,
                P, bin_capacity, alg, pk);
    BlobPlan bp = plan_blob(n, P, pk.K, ens->num_features, ens->num_groups, dtype, maxlen);
    bp.m.flags = pk.sorted ? GTS_MODEL_SORTED_BINS : 0;
    *model = bp.m;
    if (po != nullptr) {
      // the plan: per path its turns and its root's element offset, per tree
      // its first path, the bins' element ranges and the groups' bin ranges
      if (ens->num_nodes >= INT32_MAX || P >= INT32_MAX)
        return fail(GTS_EINVAL, "too many nodes or paths for a plan's 32-bit indices");
      gts_plan& pl = *po->plan;
      std::memset(&pl, 0, sizeof(pl));
      pl.num_paths = P;
      pl.num_trees = T;
      pl.num_bins = pk.K;
      pl.num_nodes = ens->num_nodes;
      for (int64_t t = 0; t < T; ++t)
        if (trees[(size_t)t].too_deep)
          return fail(GTS_EINVAL, "tree %lld: a path of more than 64 splits (a plan records "
                      "each path's turns in 64 bits)", (long long)t);
      const int64_t sizes[5] = {8 * P, 4 * P, 4 * (T + 1), 4 * (pk.K + 1),
                                4 * ((int64_t)ens->num_groups + 1)};
      int64_t cur = 0;
      for (int k = 0; k < 5; ++k) {
        pl.off[k] = cur;
        cur += (sizes[k] + kBlobAlign - 1) / kBlobAlign * kBlobAlign;
      }
      pl.bytes = cur;
      if (po->host_plan == nullptr) return GTS_OK;
      if (po->capacity < pl.bytes)
        return fail(GTS_EBUFSIZE, "plan capacity %lld < %lld bytes", (long long)po->capacity,
                    (long long)pl.bytes);
      char* hp = po->host_plan;
      // every entry of the five arrays is written below: clear only the
      // alignment gaps after each one
      for (int k = 0; k < 5; ++k) {
        const int64_t end = pl.off[k] + sizes[k];
        const int64_t next = k < 4 ? pl.off[k + 1] : pl.bytes;
        std::memset(hp + end, 0, (size_t)(next - end));
      }
      uint64_t* path_dirs = reinterpret_cast<uint64_t*>(hp + pl.off[0]);
      int32_t* path_dest = reinterpret_cast<int32_t*>(hp + pl.off[1]);
      int32_t* tree_paths = reinterpret_cast<int32_t*>(hp + pl.off[2]);
      const std::vector<Fill>& fills = pk.fills;
      const int64_t nf = (int64_t)fills.size();
      {
        // every placement's element offset, then every path's
        std::vector<int32_t>& d_at = sc.d_at;
        d_at.resize((size_t)P);
        std::atomic<int64_t> next{0};
        const int64_t step = std::max<int64_t>(1024, nf / (4 * nthreads) + 1);
        Pool::get().run(nthreads, [&]() {
          for (int64_t f0; (f0 = next.fetch_add(step)) < nf;) {
            const int64_t f1 = std::min(nf, f0 + step);
            for (int64_t f = f0; f < f1; ++f) {
              const Fill& fl = fills[(size_t)f];
              const int64_t b0 = pk.bin_offsets[(size_t)fl.b] + fl.w;
              for (int32_t i = 0; i < fl.n; ++i)
                d_at[(size_t)(fl.k + i)] = (int32_t)(b0 + (int64_t)i * fl.s);
            }
          }
        });
        std::atomic<int64_t> nt{0};
        Pool::get().run(nthreads, [&]() {
          for (int64_t t; (t = nt.fetch_add(8)) < T;) {
            for (int64_t u = t; u < std::min(T, t + 8); ++u) {
              const TreeOut& tr = trees[(size_t)u];
              int64_t p = tree_first[(size_t)u];
              tree_paths[u] = (int32_t)p;
              for (size_t j = 0; j < tr.dirs.size(); ++j, ++p) {
                path_dirs[p] = tr.dirs[j];
                path_dest[p] = d_at[(size_t)kpos[(size_t)p]];
              }
            }
          }
        });
      }
      tree_paths[T] = (int32_t)P;
      int32_t* bstart = reinterpret_cast<int32_t*>(hp + pl.off[3]);
      int32_t* gbins = reinterpret_cast<int32_t*>(hp + pl.off[4]);
      for (int64_t b = 0; b <= pk.K; ++b) bstart[b] = (int32_t)pk.bin_offsets[(size_t)b];
      for (int64_t g = 0; g <= ens->num_groups; ++g) gbins[g] = 0;
      for (int64_t b = 0; b < pk.K; ++b) gbins[pk.bin_group[(size_t)b] + 1] += 1;
      for (int64_t g = 0; g < ens->num_groups; ++g) gbins[g + 1] += gbins[g];
      return GTS_OK;
    }
    if (sizes_only) return GTS_OK;
    if (host_blob != nullptr && blob_capacity < bp.m.bytes)
      return fail(GTS_EBUFSIZE, "blob_capacity %lld < %lld bytes", (long long)blob_capacity,
                  (long long)bp.m.bytes);
    char* blob = static_cast<char*>(host_blob);
    if (direct) {
      // every placement's element offset in the blob, from the fills
      std::vector<int32_t>& d_at = sc.d_at;
      d_at.resize((size_t)P);
      {
        const std::vector<Fill>& fills = pk.fills;
        const int64_t nf = (int64_t)fills.size();
        std::atomic<int64_t> next{0};
        const int64_t step = std::max<int64_t>(1024, nf / (4 * nthreads) + 1);
        Pool::get().run(nthreads, [&]() {
          for (int64_t f0; (f0 = next.fetch_add(step)) < nf;) {
            const int64_t f1 = std::min(nf, f0 + step);
            for (int64_t f = f0; f < f1; ++f) {
              const Fill& fl = fills[(size_t)f];
              const int64_t b0 = pk.bin_offsets[(size_t)fl.b] + fl.w;
              for (int32_t i = 0; i < fl.n; ++i)
                d_at[(size_t)(fl.k + i)] = (int32_t)(b0 + (int64_t)i * fl.s);
            }
          }
        });
      }
      zero_padding(bp, blob);
      // the second walk: each leaf's path to its place, and the tree's
      // bias terms in path order
      for_each_tree(ens, status, [&](int64_t t, Walker& w) {
        TreeOut& out = trees[(size_t)t];
        out.term_sum = 0.0;
        const int64_t base = ens->tree_node_offsets[t];
        int64_t p = tree_first[(size_t)t];
        return w.walk<true, false>(ens, t, [&](int32_t leaf, size_t m) {
          const double v = ens->value[base + leaf];
          const int64_t d = d_at[(size_t)kpos[(size_t)p++]];
          const double prod = dtype == GTS_F64 ? put_path<double>(bp.m, blob, w, m, v, d)
                                               : put_path<float>(bp.m, blob, w, m, v, d);
          out.term_sum = out.term_sum + v * prod;
        });
      });
      for (int64_t t = 0; t < T; ++t)
        if (status[(size_t)t] != GTS_OK) return status[(size_t)t];
    }
    // bias: per-tree sums of the terms in path order, then per group in tree
    // order
    std::vector<double> bsum((size_t)ens->num_groups, 0.0);
    for (int64_t t = 0; t < T; ++t)
      bsum[(size_t)ens->tree_group[t]] = bsum[(size_t)ens->tree_group[t]] +
                                         trees[(size_t)t].term_sum;
    if (bias)
      for (int32_t g = 0; g < ens->num_groups; ++g) bias[g] = bsum[(size_t)g];
    if (blob && !direct) {
      zero_padding(bp, blob);
      const int64_t K = pk.K;
      // each bin's paths in placement order, with their offsets in the bin
      std::vector<PathSrc>& src_by_bin = sc.src_by_bin;
      src_by_bin.resize((size_t)P);
      {
        const std::vector<Fill>& fills = pk.fills;
        const int64_t nf = (int64_t)fills.size();
        std::atomic<int64_t> next{0};
        const int64_t step = std::max<int64_t>(1024, nf / (4 * nthreads) + 1);
        Pool::get().run(nthreads, [&]() {
          for (int64_t f0; (f0 = next.fetch_add(step)) < nf;) {
            const int64_t f1 = std::min(nf, f0 + step);
            for (int64_t f = f0; f < f1; ++f) {
              const Fill& fl = fills[(size_t)f];
              PathSrc* dst = src_by_bin.data() + pk.bin_first[(size_t)fl.b] + fl.slot;
              for (int32_t i = 0; i < fl.n; ++i) {
                PathSrc ps = src_at[(size_t)(fl.k + i)];
                ps.within = fl.w + i * fl.s;
                dst[i] = ps;
              }
            }
          }
        });
      }
      std::atomic<int64_t> next{0};
      // about eight chunks a thread, at most 64 bins each
      const int64_t chunk = std::max<int64_t>(1, std::min<int64_t>(64, K / (8 * nthreads)));
      Pool::get().run(nthreads, [&]() {
        std::vector<uint64_t> used((size_t)ens->num_features, 0);
        std::vector<int32_t> touched;
        for (;;) {
          const int64_t b0 = next.fetch_add(chunk);
          if (b0 >= K) break;
          const int64_t b1 = std::min(K, b0 + chunk);
          for (int64_t b = b0; b < b1; ++b) {
            if (dtype == GTS_F64)
              write_bin<double>(bp.m, blob, pk, src_by_bin.data(), P, b, used, touched);
            else
              write_bin<float>(bp.m, blob, pk, src_by_bin.data(), P, b, used, touched);
          }
        }
      });
    }
    if (blob)
      write_bins_and_bias(bp, blob, pk.bin_offsets.data(), pk.bin_group.data(), bsum.data());
    return GTS_OK;
  } catch (const std::bad_alloc&) {
    return fail(GTS_ENOMEM, "host allocation failed");
  }
}

}  // namespace
}  // namespace gts

extern "C" gts_status gts_prepare_model(const gts_ensemble* ens, int32_t bin_capacity,
                                        int32_t alg, int32_t dtype, gts_model* model,
                                        void* host_blob, int64_t blob_capacity, double* bias) {
  return gts::prepare_model(ens, bin_capacity, alg, dtype, model, host_blob, blob_capacity, bias,
                            nullptr);
}

extern "C" gts_status gts_plan_model(const gts_ensemble* ens, int32_t bin_capacity, int32_t alg,
                                     int32_t dtype, gts_model* model, gts_plan* plan,
                                     void* host_plan, int64_t capacity) {
  using namespace gts;
  clear_error();
  if (plan == nullptr) return fail(GTS_EINVAL, "plan must not be NULL");
  if (capacity < 0 || (capacity > 0 && host_plan == nullptr))
    return fail(GTS_EINVAL, "bad host_plan / capacity");
  const PlanOut po{plan, static_cast<char*>(host_plan), capacity};
  return prepare_model(ens, bin_capacity, alg, dtype, model, nullptr, 0, nullptr, &po);
}
