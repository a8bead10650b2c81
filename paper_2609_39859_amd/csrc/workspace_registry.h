// Library-managed device workspaces, one per (device, stream).
//
// Calls that pass no workspace of their own use the buffer of the (device,
// stream) pair they are enqueued on.  Work on one stream runs in order, so
// consecutive calls on a stream may share its buffer; calls on different
// streams get different buffers and may overlap freely.
//
// A buffer that must grow is not freed: its old allocation is retired (work
// already enqueued on the stream may still read it) and released only by
// release_all(), after the devices have been synchronised.  Growth is
// geometric (at least 1.5x, in 2 MiB granules), so the retired allocations
// of a key never hold more than twice its current one.
//
// The registry holds no HIP code: allocation, freeing and synchronisation are
// the Backend's static functions
//   int  Backend::alloc(int dev, size_t bytes, void** out)   // 0 = success
//   void Backend::free(int dev, void* p)
//   void Backend::sync(int dev)
// so that its bookkeeping can be tested on a host without a GPU.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <mutex>
#include <vector>

namespace fork {

template <class Backend>
class WorkspaceRegistry {
 public:
  static constexpr size_t kGranule = size_t(2) << 20;

  struct Slot {
    int dev;
    uintptr_t stream;
    void* ptr;
    size_t bytes;
  };

  // Buffer of (dev, stream) with at least `need` bytes.  On success *lock
  // holds the registry's mutex: the caller keeps it until its kernels are
  // enqueued, so that release_all() cannot free the buffer in between.
  // Returns 0, or the Backend's non-zero code when an allocation failed
  // (the key then keeps its previous buffer).
  int acquire(int dev, uintptr_t stream, size_t need, void** out,
              std::unique_lock<std::mutex>* lock) {
    *lock = std::unique_lock<std::mutex>(mu_);
    Slot* s = find(dev, stream);
    if (!s) {
      slots_.push_back(Slot{dev, stream, nullptr, 0});
      s = &slots_.back();
    }
    if (s->bytes < need) {
      size_t want = s->bytes + s->bytes / 2;
      if (want < need) want = need;
      want = (want + kGranule - 1) / kGranule * kGranule;
      void* p = nullptr;
      const int rc = Backend::alloc(dev, want, &p);
      if (rc != 0) {
        lock->unlock();
        return rc;
      }
      if (s->ptr) retired_.push_back(Slot{dev, stream, s->ptr, s->bytes});
      s->ptr = p;
      s->bytes = want;
    }
    *out = s->ptr;
    return 0;
  }

  // Synchronise every device that holds a buffer, then free all of them.
  void release_all() {
    std::lock_guard<std::mutex> g(mu_);
    std::vector<int> devs;
    for (const Slot& s : slots_) add_dev(&devs, s.dev);
    for (const Slot& s : retired_) add_dev(&devs, s.dev);
    for (int dev : devs) Backend::sync(dev);
    for (const Slot& s : slots_)
      if (s.ptr) Backend::free(s.dev, s.ptr);
    for (const Slot& s : retired_) Backend::free(s.dev, s.ptr);
    slots_.clear();
    retired_.clear();
  }

  // Bookkeeping, for tests: live buffers and retired allocations.
  size_t live_count() {
    std::lock_guard<std::mutex> g(mu_);
    return slots_.size();
  }
  size_t retired_count() {
    std::lock_guard<std::mutex> g(mu_);
    return retired_.size();
  }
  size_t bytes_of(int dev, uintptr_t stream) {
    std::lock_guard<std::mutex> g(mu_);
    const Slot* s = find(dev, stream);
    return s ? s->bytes : 0;
  }

 private:
  Slot* find(int dev, uintptr_t stream) {
    for (Slot& s : slots_)
      if (s.dev == dev && s.stream == stream) return &s;
    return nullptr;
  }
  static void add_dev(std::vector<int>* devs, int dev) {
    for (int d : *devs)
      if (d == dev) return;
    devs->push_back(dev);
  }

  std::mutex mu_;
  std::vector<Slot> slots_;    // one per (device, stream) key
  std::vector<Slot> retired_;  // outgrown allocations, freed by release_all
};

}  // namespace fork
