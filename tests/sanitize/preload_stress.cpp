// ThreadSanitizer stress of the preloader (host code only, plain memory pool):
// several threads hint, fetch, check and release chunk files at random while
// two more hold file sets through the restore-side interface (hold, take each
// image as it is staged, unhold) and one keeps hinting a lookahead. Every image
// a thread receives must equal its file. Exits 0 when all checks pass and no
// hold is left; the sanitizer reports data races itself.
//   usage: preload_stress <dir> [n_slots reserve max_file_kib slot_kib]
#include <atomic>
#include <chrono>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <random>
#include <string>
#include <thread>
#include <unordered_set>
#include <vector>

#include "kvx.h"
#include "kvx_preload.h"

int main(int argc, char** argv) {
  if (argc < 2) return 2;
  const int n_files = 24;
  const int n_slots = argc > 2 ? atoi(argv[2]) : 10;
  const int reserve = argc > 3 ? atoi(argv[3]) : 2;
  const size_t max_file = (size_t)(argc > 4 ? atoi(argv[4]) : 1536) << 10;
  const int64_t slot = (int64_t)(argc > 5 ? atoi(argv[5]) : 2048) << 10;
  std::vector<std::string> paths;
  std::vector<std::vector<unsigned char>> data;
  std::mt19937 rng(1);
  for (int i = 0; i < n_files; ++i) {
    std::string p = std::string(argv[1]) + "/f" + std::to_string(i);
    std::vector<unsigned char> d(4096 + rng() % max_file);
    for (auto& b : d) b = (unsigned char)rng();
    FILE* f = fopen(p.c_str(), "wb");
    if (!f || fwrite(d.data(), 1, d.size(), f) != d.size()) return 3;
    fclose(f);
    paths.push_back(p);
    data.push_back(std::move(d));
  }
  kvx_preloader* pre = nullptr;
  if (kvx_preloader_create(n_slots, slot, 4, reserve, 0, &pre) != KVX_OK) return 4;
  std::atomic<int> bad{0};
  auto same = [&](const void* img, int64_t size, int i) {
    return (size_t)size == data[(size_t)i].size() && memcmp(img, data[(size_t)i].data(), (size_t)size) == 0;
  };
  std::vector<std::thread> th;
  for (int t = 0; t < 4; ++t)
    th.emplace_back([&, t] {  // request-like threads: hint a few, fetch two, release
      std::mt19937 r(100 + t);
      for (int it = 0; it < 50; ++it) {
        const char* hint[4];
        for (auto& h : hint) h = paths[r() % n_files].c_str();
        kvx_preload_hint(pre, hint, 4);
        int idx[2] = {(int)(r() % n_files), (int)(r() % n_files)};
        const char* want[2] = {paths[(size_t)idx[0]].c_str(), paths[(size_t)idx[1]].c_str()};
        void* img[2];
        int64_t sz[2];
        const kvx_status st = kvx_preload_fetch(pre, want, 2, img, sz);
        if (st == KVX_ENOMEM) continue;
        if (st != KVX_OK) {
          ++bad;
          continue;
        }
        for (int k = 0; k < 2; ++k)
          if (!same(img[k], sz[k], idx[k])) ++bad;
        if (kvx_preload_release(pre, want, 2) != KVX_OK) ++bad;
        std::this_thread::sleep_for(std::chrono::microseconds(300 + r() % 1500));
      }
    });
  for (int t = 0; t < 2; ++t)
    th.emplace_back([&, t] {  // restore-like holders: hold a set, take images as staged
      std::mt19937 r(300 + t);
      std::atomic<bool> cancel{false};
      for (int it = 0; it < 30; ++it) {
        std::vector<std::string> want;
        std::vector<int> idx;
        std::unordered_set<int> seen;
        for (int k = 0; k < 3; ++k) {
          const int i = (int)(r() % n_files);
          if (seen.insert(i).second) {
            idx.push_back(i);
            want.push_back(paths[(size_t)i]);
          }
        }
        std::vector<void*> holds;
        const kvx_status st = kvx::preload_hold(pre, want, &holds);
        if (st == KVX_ENOMEM) continue;
        if (st != KVX_OK) {
          ++bad;
          continue;
        }
        for (size_t k = 0; k < holds.size(); ++k) {
          uint8_t* img = nullptr;
          int64_t size = 0;
          kvx_status s2 = kvx::preload_image(pre, holds[k], false, &cancel, &img, &size);
          if (s2 == KVX_OK && !img) s2 = kvx::preload_image(pre, holds[k], true, &cancel, &img, &size);
          if (s2 != KVX_OK || !img || !same(img, size, idx[k])) ++bad;
        }
        kvx::preload_unhold(pre, holds);
      }
    });
  th.emplace_back([&] {  // a scheduler's lookahead over its waiting queue
    std::mt19937 r(7);
    for (int it = 0; it < 300; ++it) {
      const char* h[2] = {paths[r() % n_files].c_str(), paths[r() % n_files].c_str()};
      kvx_preload_hint(pre, h, 2);
      std::this_thread::sleep_for(std::chrono::microseconds(150));
    }
  });
  for (auto& x : th) x.join();
  kvx_preload_wait_idle(pre);
  kvx_preload_stats s{};
  kvx_preload_stats_get(pre, &s);
  printf("bad %d fetches %lld reads %lld/%lld hits %lld/%lld evictions %lld preempted %lld held %lld\n",
         bad.load(), (long long)s.demand_fetches, (long long)s.spec_reads, (long long)s.demand_reads,
         (long long)s.hits_ready, (long long)s.hits_inflight, (long long)s.evictions,
         (long long)s.spec_preempted, (long long)s.held);
  kvx_preloader_destroy(pre);
  return bad.load() != 0 || s.held != 0 ? 1 : 0;
}
