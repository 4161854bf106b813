// Host-only checks of the descriptor-table cache policy
// (paper_2607_10611_amd/csrc/table_cache.h) with a fake backend that records
// every allocation, free, upload, event record and host wait.  Built and run
// by tests/test_table_cache.py; prints "ok" and exits 0 when every check holds.
#include <stdio.h>
#include <stdlib.h>

#include <string>
#include <vector>

#include "table_cache.h"

namespace {

struct Op {
  std::string kind;  // alloc, free, upload, record, wait
  void* mem;
  int event;
};

struct Fake {
  using Event = int;
  std::vector<Op> log;
  uintptr_t next = 0x1000;
  int next_event = 0;
  bool fail_alloc = false;
  bool alloc(size_t bytes, void** p) {
    if (fail_alloc) return false;
    *p = (void*)next;
    next += (bytes + 0xFFF) & ~(size_t)0xFFF;
    log.push_back({"alloc", *p, -1});
    return true;
  }
  void free(void* p) { log.push_back({"free", p, -1}); }
  bool upload(void* dst, const void*, size_t, void*) {
    log.push_back({"upload", dst, -1});
    return true;
  }
  bool new_event(Event* e) {
    *e = next_event++;
    return true;
  }
  bool record(Event e, void*) {
    log.push_back({"record", nullptr, e});
    return true;
  }
  bool wait(Event e) {
    log.push_back({"wait", nullptr, e});
    return true;
  }
  size_t count(const char* k, void* mem = nullptr) const {
    size_t n = 0;
    for (const Op& o : log)
      if (o.kind == k && (!mem || o.mem == mem)) ++n;
    return n;
  }
};

int failures = 0;
#define CHECK(c)                                                  \
  do {                                                            \
    if (!(c)) {                                                   \
      fprintf(stderr, "%s:%d: check failed: %s\n", __FILE__, __LINE__, #c); \
      ++failures;                                                 \
    }                                                             \
  } while (0)

using Cache = madd_cache::TableCache<Fake>;

// A table of `ndesc` 88-byte descriptors whose bytes identify list `id`.
std::vector<uint8_t> table(int id, int ndesc = 3) {
  std::vector<uint8_t> t((size_t)ndesc * 88, 0);
  for (size_t i = 0; i < t.size(); i += 8) t[i] = (uint8_t)(id * 7 + i);
  t[1] = (uint8_t)id;
  t[2] = (uint8_t)(id >> 8);
  return t;
}

// One eager step of list `id`: acquire, "launch", release.
void* eager(Cache& c, Fake& f, int id, int device = 0, int ndesc = 3) {
  const std::vector<uint8_t> t = table(id, ndesc);
  void* mem = nullptr;
  size_t slot = 0;
  CHECK(c.acquire(f, device, t.data(), t.size(), false, nullptr, &mem, &slot) == madd_cache::kOk);
  CHECK(c.release(f, slot, false, nullptr, true) == madd_cache::kOk);
  return mem;
}

void hit_uploads_nothing() {
  Cache c;
  Fake f;
  void* a = eager(c, f, 1);
  void* b = eager(c, f, 1);
  CHECK(a == b);
  CHECK(f.count("upload") == 1 && f.count("alloc") == 1);
  CHECK(f.count("record") == 2 && f.count("wait") == 0);
}

void lru_is_recycled_after_its_event() {
  Cache c;
  Fake f;
  std::vector<void*> mem;
  for (int id = 0; id < 32; ++id) mem.push_back(eager(c, f, id));
  eager(c, f, 0);  // list 0 is now the most recent; list 1 is the LRU
  const size_t allocs = f.count("alloc");
  f.log.clear();
  void* m = eager(c, f, 100);
  CHECK(m == mem[1]);              // list 1's memory, reused
  CHECK(f.count("alloc") == 0 && f.count("free") == 0 && allocs == 32);
  CHECK(f.log.size() >= 2 && f.log[0].kind == "wait" && f.log[1].kind == "upload");
  CHECK(f.log[1].mem == mem[1]);   // the wait comes before the overwrite
  f.log.clear();
  void* again = eager(c, f, 1);    // list 1 was evicted: uploaded anew
  CHECK(f.count("upload") == 1 && again != nullptr);
  CHECK(c.size() == 32);
}

void pinned_table_survives_forty_lists() {
  Cache c;
  Fake f;
  void* p = eager(c, f, 7);
  // the same list while the stream is capturing: a hit, pinned
  const std::vector<uint8_t> t = table(7);
  void* mem = nullptr;
  size_t slot = 0;
  f.log.clear();
  CHECK(c.acquire(f, 0, t.data(), t.size(), true, nullptr, &mem, &slot) == madd_cache::kOk);
  CHECK(c.release(f, slot, true, nullptr, true) == madd_cache::kOk);
  CHECK(mem == p && f.log.empty());   // nothing allocated, uploaded or recorded
  CHECK(c.pinned() == 1);
  for (int id = 200; id < 240; ++id) eager(c, f, id);
  CHECK(f.count("upload", p) == 0 && f.count("free", p) == 0);
  f.log.clear();
  CHECK(eager(c, f, 7) == p);
  CHECK(f.count("upload") == 0);
  CHECK(c.size() == 33);              // 32 unpinned + the pinned one
}

void capture_miss_is_refused_without_side_effects() {
  Cache c;
  Fake f;
  eager(c, f, 1);
  f.log.clear();
  const std::vector<uint8_t> t = table(9);
  void* mem = nullptr;
  size_t slot = 0;
  CHECK(c.acquire(f, 0, t.data(), t.size(), true, nullptr, &mem, &slot) ==
        madd_cache::kCaptureMiss);
  CHECK(f.log.empty() && mem == nullptr && c.size() == 1);
}

void small_victim_is_freed_after_its_event() {
  Cache c;
  Fake f;
  std::vector<void*> mem;
  for (int id = 0; id < 32; ++id) mem.push_back(eager(c, f, id, 0, 3));
  f.log.clear();
  void* big = eager(c, f, 500, 0, 300);  // 300 descriptors: more than a 64-descriptor slot
  CHECK(big != mem[0]);
  CHECK(f.log.size() >= 4 && f.log[0].kind == "wait" && f.log[1].kind == "free" &&
        f.log[1].mem == mem[0] && f.log[2].kind == "alloc" && f.log[3].kind == "upload");
}

void held_tables_are_not_recycled() {
  Cache c;
  Fake f;
  std::vector<size_t> slots;
  for (int id = 0; id < 32; ++id) {
    const std::vector<uint8_t> t = table(id);
    void* mem = nullptr;
    size_t slot = 0;
    CHECK(c.acquire(f, 0, t.data(), t.size(), false, nullptr, &mem, &slot) == madd_cache::kOk);
    slots.push_back(slot);
  }
  f.log.clear();
  eager(c, f, 77);  // every table is held: the cache grows
  CHECK(f.count("wait") == 0 && f.count("alloc") == 1 && c.size() == 33);
  for (size_t s : slots) CHECK(c.release(f, s, false, nullptr, false) == madd_cache::kOk);
  CHECK(f.count("record") == 1);  // only list 77 launched
}

void devices_are_separate() {
  Cache c;
  Fake f;
  for (int id = 0; id < 32; ++id) eager(c, f, id, 0);
  f.log.clear();
  eager(c, f, 0, 1);  // same bytes, other device: a miss there, no eviction here
  CHECK(f.count("wait") == 0 && f.count("alloc") == 1 && c.size() == 33);
  f.log.clear();
  eager(c, f, 0, 0);  // still cached on device 0
  CHECK(f.count("upload") == 0);
}

void failed_allocation_leaves_a_usable_cache() {
  Cache c;
  Fake f;
  f.fail_alloc = true;
  const std::vector<uint8_t> t = table(3);
  void* mem = nullptr;
  size_t slot = 0;
  CHECK(c.acquire(f, 0, t.data(), t.size(), false, nullptr, &mem, &slot) == madd_cache::kNoMem);
  f.fail_alloc = false;
  CHECK(eager(c, f, 3) != nullptr);
}

}  // namespace

int main() {
  hit_uploads_nothing();
  lru_is_recycled_after_its_event();
  pinned_table_survives_forty_lists();
  capture_miss_is_refused_without_side_effects();
  small_victim_is_freed_after_its_event();
  held_tables_are_not_recycled();
  devices_are_separate();
  failed_allocation_leaves_a_usable_cache();
  if (failures) {
    fprintf(stderr, "%d check(s) failed\n", failures);
    return 1;
  }
  printf("ok\n");
  return 0;
}
