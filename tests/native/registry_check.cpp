// Host-only checks of the workspace registry's bookkeeping (keying by
// (device, stream), geometric growth, retirement of outgrown buffers, release
// after synchronising every device), with a fake backend that records calls.
#include <stdio.h>
#include <stdlib.h>

#include <string>
#include <thread>
#include <vector>

#include "workspace_registry.h"

namespace {

std::vector<std::string> g_log;
int g_fail_next = 0;
char g_heap[1 << 12];
size_t g_used = 0;

struct FakeBackend {
  static int alloc(int dev, size_t bytes, void** out) {
    if (g_fail_next) {
      g_fail_next = 0;
      return -4;
    }
    *out = g_heap + (g_used++ % sizeof g_heap);
    g_log.push_back("alloc " + std::to_string(dev) + " " + std::to_string(bytes));
    return 0;
  }
  static void free(int dev, void* p) {
    (void)p;
    g_log.push_back("free " + std::to_string(dev));
  }
  static void sync(int dev) { g_log.push_back("sync " + std::to_string(dev)); }
};

int g_errors = 0;
#define CHECK(c)                                                 \
  do {                                                           \
    if (!(c)) {                                                  \
      fprintf(stderr, "FAILED line %d: %s\n", __LINE__, #c);    \
      ++g_errors;                                                \
    }                                                            \
  } while (0)

}  // namespace

int main() {
  using Reg = fork::WorkspaceRegistry<FakeBackend>;
  const size_t MiB = size_t(1) << 20;
  Reg reg;
  void *a = nullptr, *b = nullptr, *c = nullptr, *a2 = nullptr;
  std::unique_lock<std::mutex> lk;

  // distinct streams of one device get distinct buffers
  CHECK(reg.acquire(0, 0x10, 3 * MiB, &a, &lk) == 0 && lk.owns_lock());
  lk.unlock();
  CHECK(reg.acquire(0, 0x20, 1, &b, &lk) == 0);
  lk.unlock();
  CHECK(a != b);
  CHECK(reg.live_count() == 2);
  CHECK(reg.bytes_of(0, 0x10) == 4 * MiB);  // rounded to 2 MiB granules
  CHECK(reg.bytes_of(0, 0x20) == 2 * MiB);
  // the same stream on another device is another key
  CHECK(reg.acquire(1, 0x10, 1, &c, &lk) == 0);
  lk.unlock();
  CHECK(reg.live_count() == 3 && c != a);
  // a request that fits reuses the buffer without allocating
  const size_t nlog = g_log.size();
  CHECK(reg.acquire(0, 0x10, 4 * MiB, &a2, &lk) == 0);
  lk.unlock();
  CHECK(a2 == a && g_log.size() == nlog);
  // growth: at least 1.5x, the old buffer retired (not freed)
  CHECK(reg.acquire(0, 0x10, 4 * MiB + 1, &a2, &lk) == 0);
  lk.unlock();
  CHECK(reg.bytes_of(0, 0x10) == 6 * MiB);
  CHECK(reg.retired_count() == 1);
  CHECK(g_log.back() == "alloc 0 " + std::to_string(6 * MiB));
  // a large jump allocates what is needed
  CHECK(reg.acquire(0, 0x10, 40 * MiB, &a2, &lk) == 0);
  lk.unlock();
  CHECK(reg.bytes_of(0, 0x10) == 40 * MiB && reg.retired_count() == 2);
  // a failed allocation keeps the previous buffer and releases the lock
  g_fail_next = 1;
  void* d = nullptr;
  CHECK(reg.acquire(0, 0x10, 100 * MiB, &d, &lk) == -4);
  CHECK(!lk.owns_lock());
  CHECK(reg.bytes_of(0, 0x10) == 40 * MiB && reg.retired_count() == 2);
  // concurrent acquisitions from host threads on their own streams
  std::vector<std::thread> ts;
  std::vector<void*> got(8, nullptr);
  for (int t = 0; t < 8; ++t)
    ts.emplace_back([&, t] {
      std::unique_lock<std::mutex> l;
      void* p = nullptr;
      if (reg.acquire(2, 0x100 + t, (t + 1) * MiB, &p, &l) == 0) got[t] = p;
    });
  for (auto& t : ts) t.join();
  for (int t = 0; t < 8; ++t) CHECK(got[t] != nullptr && reg.bytes_of(2, 0x100 + t) >= (t + 1) * MiB);
  CHECK(reg.live_count() == 11);
  // release: every device synchronised before anything is freed
  g_log.clear();
  reg.release_all();
  size_t syncs = 0, frees = 0;
  bool order_ok = true;
  for (const std::string& s : g_log) {
    if (s.rfind("sync", 0) == 0) {
      ++syncs;
      if (frees) order_ok = false;
    } else if (s.rfind("free", 0) == 0) {
      ++frees;
    }
  }
  CHECK(syncs == 3);        // devices 0, 1, 2
  CHECK(frees == 11 + 2);   // live buffers + retired allocations
  CHECK(order_ok);
  CHECK(reg.live_count() == 0 && reg.retired_count() == 0);
  // usable again after release
  CHECK(reg.acquire(0, 0x10, 1, &a, &lk) == 0);
  lk.unlock();
  CHECK(reg.live_count() == 1);
  if (g_errors) return 1;
  printf("registry ok\n");
  return 0;
}
