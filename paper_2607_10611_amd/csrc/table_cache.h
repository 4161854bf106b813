// Cache of device descriptor tables for multi-tensor steps: the policy,
// free of HIP so that it can be exercised on the host with a fake backend.
//
// A multi-tensor step launches its kernels with a device table that lists
// the tensors (pointers, sizes, index bases).  Lists repeat from one training
// step to the next, so tables are kept by content and a repeated list enqueues
// only its kernels.  Rules:
//   - A hit returns the cached device table; nothing is uploaded.
//   - A miss uploads the table asynchronously on the caller's stream (the
//     backend's upload is stream-ordered, so the launches that follow on that
//     stream see it).  Any later step of the same tensors must already be
//     ordered after this one by the caller (both update the same buffers), so
//     it is ordered after the upload as well.
//   - At most kMaxUnpinned unpinned tables per device.  On a miss past that
//     limit the least recently used unpinned table is recycled: the host
//     waits for the event recorded after that table's last launch (only that
//     launch, not the device), then reuses its memory when large enough, or
//     frees it and allocates anew.  A table between acquire() and release()
//     (its launches not yet enqueued) is never recycled; when every table is
//     pinned or held the cache grows instead.
//   - A table hit while the caller's stream is capturing a graph is pinned:
//     the graph holds its address, so it is never recycled or freed.
//   - A miss while capturing is refused (kCaptureMiss): allocating, uploading
//     or waiting inside a capture would break it or record work the replays
//     repeat.  The caller steps the list once outside the capture first.
//   - Events are recorded only outside captures (pinned tables need none).
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
//   using Event = ...;                      copyable handle
//   bool alloc(size_t bytes, void** p);     device memory on the current device
//   void free(void* p);
//   bool upload(void* dst, const void* src, size_t bytes, void* stream);  async, stream-ordered
//   bool new_event(Event* e);
//   bool record(Event e, void* stream);
//   bool wait(Event e);                     host waits until e has completed
template <class Backend>
class TableCache {
 public:
  static constexpr size_t kMaxUnpinned = 32;
  static constexpr size_t kGranule = 64 * 88;  // capacity rounding (64 descriptors)

  struct Entry {
    int device;
    std::vector<uint8_t> key;  // the table's bytes
    void* mem;
    size_t cap;
    uint64_t last_use;
    bool pinned;
    bool has_event;
    int holds;  // acquire() calls not yet released
    typename Backend::Event ev;
  };

  // The device table for `bytes`; `*slot` identifies the entry, which the
  // caller passes to release() once the launches reading it are enqueued
  // (or have failed).  Entries are never removed, so a slot stays valid.
  int acquire(Backend& be, int device, const void* bytes, size_t nbytes, bool capturing,
              void* stream, void** out, size_t* slot) {
    std::lock_guard<std::mutex> lock(mu_);
    ++clock_;
    for (size_t i = 0; i < entries_.size(); ++i) {
      Entry& e = entries_[i];
      if (e.device == device && e.key.size() == nbytes && memcmp(e.key.data(), bytes, nbytes) == 0) {
        e.last_use = clock_;
        if (capturing) e.pinned = true;
        ++e.holds;
        *out = e.mem;
        *slot = i;
        return kOk;
      }
    }
    if (capturing) return kCaptureMiss;
    const size_t cap = (nbytes + kGranule - 1) / kGranule * kGranule;
    size_t unpinned = 0, victim = entries_.size();
    for (size_t i = 0; i < entries_.size(); ++i) {
      const Entry& e = entries_[i];
      if (e.device != device || e.pinned) continue;
      ++unpinned;
      if (e.holds > 0) continue;
      if (victim == entries_.size() || e.last_use < entries_[victim].last_use) victim = i;
    }
    size_t idx;
    if (unpinned >= kMaxUnpinned && victim < entries_.size()) {
      Entry& v = entries_[victim];
      if (v.has_event && !be.wait(v.ev)) return kDevice;
      v.has_event = false;
      v.key.clear();  // matches nothing until refilled
      if (v.cap < cap) {
        be.free(v.mem);
        v.mem = nullptr;
        v.cap = 0;
        if (!be.alloc(cap, &v.mem)) {
          v.mem = nullptr;
          return kNoMem;
        }
        v.cap = cap;
      }
      idx = victim;
    } else {
      Entry e;
      e.device = device;
      e.mem = nullptr;
      e.cap = cap;
      e.pinned = false;
      e.has_event = false;
      e.holds = 0;
      if (!be.alloc(cap, &e.mem)) return kNoMem;
      if (!be.new_event(&e.ev)) {
        be.free(e.mem);
        return kDevice;
      }
      entries_.push_back(e);
      idx = entries_.size() - 1;
    }
    Entry& e = entries_[idx];
    e.last_use = clock_;
    if (!be.upload(e.mem, bytes, nbytes, stream)) return kDevice;
    e.key.assign((const uint8_t*)bytes, (const uint8_t*)bytes + nbytes);
    ++e.holds;
    *out = e.mem;
    *slot = idx;
    return kOk;
  }

  // The launches that read the table of `slot` are enqueued on `stream`
  // (launched = true) or were not (an error): outside a capture, record the
  // event a later recycling waits for.
  int release(Backend& be, size_t slot, bool capturing, void* stream, bool launched) {
    std::lock_guard<std::mutex> lock(mu_);
    if (slot >= entries_.size()) return kOk;
    Entry& e = entries_[slot];
    if (e.holds > 0) --e.holds;
    if (capturing || !launched || e.pinned) return kOk;
    if (!be.record(e.ev, stream)) return kDevice;
    e.has_event = true;
    return kOk;
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
