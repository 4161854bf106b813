// Cache of device descriptor tables for multi-tensor steps: the policy,
// free of HIP so that it can be exercised on the host with a fake backend.
//
// A multi-tensor step launches its kernels with a device table that lists
// the tensors (pointers, sizes, index bases).  Lists repeat from one training
// step to the next, so tables are kept by content and a repeated list enqueues
// only its kernels.  Rules:
//   - A hit returns the cached device table; nothing is uploaded.  The entry
//     remembers the stream of its latest use.
//   - A miss uploads the table asynchronously on the caller's stream (the
//     backend's upload is stream-ordered, so the launches that follow on that
//     stream see it).
//   - Recycling needs no event and no host wait: a table is only ever
//     recycled by a call on the stream of its latest use, so the new upload is
//     queued behind every launch that read it there.  Launches of the same
//     table on other streams came earlier and were ordered before that latest
//     one by the caller, who must order any two steps of the same tensors
//     (both update the same buffers).
//   - Up to kMaxUnpinned unpinned tables per (device, stream); a miss past that
//     recycles the least recently used idle table of that stream whose memory
//     is large enough, else it allocates a new one.  Memory is never freed,
//     so nothing ever waits for the device.
//   - A table between acquire() and release() (its launches not yet
//     enqueued) is never recycled.
//   - A table hit while the caller's stream is capturing a graph is pinned:
//     the graph holds its address, so it is never recycled.
//   - A miss while capturing is refused (kCaptureMiss): allocating or
//     uploading inside a capture would break it or add work to every replay.
//     The caller steps the list once outside the capture first.
#ifndef MADD_TABLE_CACHE_H
#define MADD_TABLE_CACHE_H

#include <stddef.h>
#include <stdint.h>
#include <string.h>

#include <mutex>
#include <vector>

namespace madd_cache {

enum Status : int { kOk = 0, kCaptureMiss = 1, kNoMem = 2, kDevice = 3 };

// Backend interface (duck-typed):
//   bool alloc(size_t bytes, void** p);     device memory on the current device
//   bool upload(void* dst, const void* src, size_t bytes, void* stream);  async, stream-ordered
template <class Backend>
class TableCache {
 public:
  static constexpr size_t kMaxUnpinned = 32;
  static constexpr size_t kMinCap = 64 * 88;  // smallest table capacity (64 descriptors)

  struct Entry {
    int device;
    uint64_t stream;           // identity of the stream of the latest use
    std::vector<uint8_t> key;  // the table's bytes; empty while being refilled
    void* mem;
    size_t cap;
    uint64_t last_use;
    bool pinned;
    int holds;  // acquire() calls not yet released
  };

  // Capacity class of a table of `bytes`: a power-of-two multiple of kMinCap.
  static size_t capacity_for(size_t bytes) {
    size_t c = kMinCap;
    while (c < bytes) c *= 2;
    return c;
  }

  // The device table for `bytes`, used on the stream identified by `stream`
  // (`stream_handle` is passed to the backend's upload).  `*slot` identifies
  // the entry, which the caller passes to release() once the launches reading
  // it are enqueued (or have failed).  Entries are never removed, so a slot
  // stays valid.
  int acquire(Backend& be, int device, uint64_t stream, const void* bytes, size_t nbytes,
              bool capturing, void* stream_handle, void** out, size_t* slot) {
    std::lock_guard<std::mutex> lock(mu_);
    ++clock_;
    for (size_t i = 0; i < entries_.size(); ++i) {
      Entry& e = entries_[i];
      if (e.device == device && e.key.size() == nbytes &&
          memcmp(e.key.data(), bytes, nbytes) == 0) {
        e.last_use = clock_;
        e.stream = stream;
        if (capturing) e.pinned = true;
        ++e.holds;
        *out = e.mem;
        *slot = i;
        return kOk;
      }
    }
    if (capturing) return kCaptureMiss;
    const size_t cap = capacity_for(nbytes);
    size_t same = 0, victim = entries_.size();
    for (size_t i = 0; i < entries_.size(); ++i) {
      const Entry& e = entries_[i];
      if (e.device != device || e.stream != stream || e.pinned) continue;
      ++same;
      if (e.holds > 0 || e.cap < cap) continue;
      if (victim == entries_.size() || e.last_use < entries_[victim].last_use) victim = i;
    }
    size_t idx;
    if (same >= kMaxUnpinned && victim < entries_.size()) {
      idx = victim;
    } else {
      Entry e;
      e.device = device;
      e.stream = stream;
      e.mem = nullptr;
      e.cap = cap;
      e.pinned = false;
      e.holds = 0;
      if (!be.alloc(cap, &e.mem)) return kNoMem;
      entries_.push_back(e);
      idx = entries_.size() - 1;
    }
    Entry& e = entries_[idx];
    e.key.clear();  // matches nothing unless the upload is enqueued
    e.last_use = clock_;
    if (!be.upload(e.mem, bytes, nbytes, stream_handle)) return kDevice;
    e.key.assign((const uint8_t*)bytes, (const uint8_t*)bytes + nbytes);
    ++e.holds;
    *out = e.mem;
    *slot = idx;
    return kOk;
  }

  // The launches that read the table of `slot` are enqueued (or failed).
  void release(size_t slot) {
    std::lock_guard<std::mutex> lock(mu_);
    if (slot < entries_.size() && entries_[slot].holds > 0) --entries_[slot].holds;
  }

  // Introspection for tests.
  size_t size() const {
    std::lock_guard<std::mutex> lock(mu_);
    return entries_.size();
  }
  size_t pinned() const {
    std::lock_guard<std::mutex> lock(mu_);
    size_t k = 0;
    for (const Entry& e : entries_) k += e.pinned ? 1 : 0;
    return k;
  }

 private:
  mutable std::mutex mu_;
  std::vector<Entry> entries_;
  uint64_t clock_ = 0;
};

}  // namespace madd_cache

#endif  // MADD_TABLE_CACHE_H
