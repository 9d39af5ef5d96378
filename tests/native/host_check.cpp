// Host-side check driver, built by tests/test_host_sanitizers.py with
// AddressSanitizer + UndefinedBehaviorSanitizer (or ThreadSanitizer) together
// with the library's host source.  It reads an ensemble from raw files in the
// current directory and, for every packing heuristic, two bin capacities and
// both dtypes, prepares the model twice (size query, then the blob) and
// compares the blob byte for byte with the three-call route
// extract -> pack -> layout.  Then six threads with different thread caps
// (gts_set_host_threads) prepare the BFD model at the same time, several
// times each, sharing the worker pool, and every blob must equal the
// one-at-a-time blob.  Exit status
// 0 only if every case matches.
#include <cstdio>
#include <cstdlib>
#include <thread>
#include <vector>

#include "gts.h"

template <typename T>
static std::vector<T> read_all(const char* name) {
  std::vector<T> v;
  FILE* f = std::fopen(name, "rb");
  if (!f) return v;
  T x;
  while (std::fread(&x, sizeof(T), 1, f) == 1) v.push_back(x);
  std::fclose(f);
  return v;
}

int main() {
  const auto hdr = read_all<int64_t>("hdr.bin");  // M, G, T, N
  if (hdr.size() != 4) return 2;
  auto off = read_all<int64_t>("off.bin");
  auto grp = read_all<int32_t>("grp.bin");
  auto left = read_all<int32_t>("left.bin"), right = read_all<int32_t>("right.bin");
  auto feat = read_all<int32_t>("feat.bin");
  auto thr = read_all<float>("thr.bin");
  auto cov = read_all<double>("cov.bin"), val = read_all<double>("val.bin");
  const gts_ensemble e{(int32_t)hdr[0], (int32_t)hdr[1], hdr[2], hdr[3], off.data(), grp.data(),
                       left.data(), right.data(), feat.data(), thr.data(), cov.data(),
                       val.data()};
  const int32_t M = (int32_t)hdr[0], G = (int32_t)hdr[1];
  int bad = 0;
  for (int alg = GTS_PACK_BFD; alg <= GTS_PACK_NONE; ++alg)
    for (int cap : {64, 17})
      for (int dt : {GTS_F32, GTS_F64}) {
        gts_model m;
        gts_status st = gts_prepare_model(&e, cap, alg, dt, &m, nullptr, 0, nullptr);
        if (st == GTS_EPATHLEN) continue;  // paths longer than this capacity
        if (st != GTS_OK) { std::printf("size query: %s\n", gts_last_error()); ++bad; continue; }
        std::vector<char> blob((size_t)m.bytes);
        std::vector<double> bias((size_t)G);
        st = gts_prepare_model(&e, cap, alg, dt, &m, blob.data(), m.bytes, bias.data());
        if (st != GTS_OK) { std::printf("prepare: %s\n", gts_last_error()); ++bad; continue; }
        int64_t n = 0, P = 0, K = 0;
        gts_extract_paths(&e, nullptr, 0, &n, &P, nullptr);
        std::vector<gts_path_element> el((size_t)n), packed((size_t)n);
        std::vector<double> bias2((size_t)G);
        gts_extract_paths(&e, el.data(), n, &n, &P, bias2.data());
        gts_pack_paths(el.data(), n, cap, alg, nullptr, nullptr, 0, &K);
        std::vector<int64_t> offs((size_t)K + 1);
        gts_pack_paths(el.data(), n, cap, alg, packed.data(), offs.data(), K + 1, &K);
        gts_model m2;
        gts_model_layout(packed.data(), n, offs.data(), K, M, G, bias2.data(), dt, &m2, nullptr, 0);
        std::vector<char> blob2((size_t)m2.bytes);
        st = gts_model_layout(packed.data(), n, offs.data(), K, M, G, bias2.data(), dt, &m2,
                              blob2.data(), m2.bytes);
        const bool same = st == GTS_OK && blob == blob2 && bias == bias2;
        std::printf("alg %d cap %d dtype %d bins %lld %s\n", alg, cap, dt, (long long)m.num_bins,
                    same ? "same" : "DIFFERENT");
        if (!same) ++bad;
      }
  for (int dt : {GTS_F32, GTS_F64}) {
    gts_model m;
    if (gts_prepare_model(&e, 64, GTS_PACK_BFD, dt, &m, nullptr, 0, nullptr) != GTS_OK) {
      ++bad;
      continue;
    }
    std::vector<char> want((size_t)m.bytes);
    std::vector<double> want_bias((size_t)G);
    gts_prepare_model(&e, 64, GTS_PACK_BFD, dt, &m, want.data(), m.bytes, want_bias.data());
    int wrong[6] = {0, 0, 0, 0, 0, 0};
    std::vector<std::thread> th;
    for (int k = 0; k < 6; ++k)
      th.emplace_back([&, k] {
        gts_set_host_threads(k == 0 ? 4 : k == 1 ? 2 : k == 2 ? 1 : 0);
        for (int r = 0; r < 4; ++r) {
          gts_model mk;
          std::vector<char> blob((size_t)m.bytes);
          std::vector<double> bias((size_t)G);
          const gts_status st = gts_prepare_model(&e, 64, GTS_PACK_BFD, dt, &mk, blob.data(),
                                                  m.bytes, bias.data());
          if (st != GTS_OK || blob != want || bias != want_bias) ++wrong[k];
        }
      });
    for (auto& t : th) t.join();
    int nwrong = 0;
    for (int k = 0; k < 6; ++k) nwrong += wrong[k];
    const bool same = nwrong == 0;
    std::printf("concurrent dtype %d %s\n", dt, same ? "same" : "DIFFERENT");
    if (!same) ++bad;
  }
  return bad == 0 ? 0 : 1;
}
