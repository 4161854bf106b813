// Host-only checks of the descriptor-table cache policy
// (paper_2607_10611_amd/csrc/table_cache.h) with a fake backend that records
// every allocation and upload.  Built and run by tests/test_table_cache.py;
// prints "ok" and exits 0 when every check holds.
#include <stdio.h>
#include <stdlib.h>

#include <string>
#include <vector>

#include "table_cache.h"

namespace {

struct Op {
  std::string kind;  // alloc, upload
  void* mem;
  void* stream;
};

struct Fake {
  std::vector<Op> log;
  uintptr_t next = 0x1000;
  bool fail_alloc = false;
  bool alloc(size_t bytes, void** p) {
    if (fail_alloc) return false;
    *p = (void*)next;
    next += (bytes + 0xFFF) & ~(size_t)0xFFF;
    log.push_back({"alloc", *p, nullptr});
    return true;
  }
  bool upload(void* dst, const void*, size_t, void* stream) {
    log.push_back({"upload", dst, stream});
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
#define CHECK(c)                                                            \
  do {                                                                      \
    if (!(c)) {                                                             \
      fprintf(stderr, "%s:%d: check failed: %s\n", __FILE__, __LINE__, #c); \
      ++failures;                                                           \
    }                                                                       \
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

void* handle(uint64_t stream) { return (void*)(uintptr_t)(0x5000 + stream); }

// One eager step of list `id` on `stream`: acquire, "launch", release.
void* eager(Cache& c, Fake& f, int id, uint64_t stream = 1, int device = 0, int ndesc = 3) {
  const std::vector<uint8_t> t = table(id, ndesc);
  void* mem = nullptr;
  size_t slot = 0;
  CHECK(c.acquire(f, device, stream, t.data(), t.size(), false, handle(stream), &mem, &slot) ==
        madd_cache::kOk);
  c.release(slot);
  return mem;
}

void hit_uploads_nothing() {
  Cache c;
  Fake f;
  void* a = eager(c, f, 1);
  void* b = eager(c, f, 1);
  CHECK(a == b);
  CHECK(f.count("upload") == 1 && f.count("alloc") == 1);
}

void lru_of_the_same_stream_is_recycled_in_stream_order() {
  Cache c;
  Fake f;
  std::vector<void*> mem;
  for (int id = 0; id < 32; ++id) mem.push_back(eager(c, f, id));
  eager(c, f, 0);  // list 0 is now the most recent; list 1 is the LRU
  f.log.clear();
  void* m = eager(c, f, 100);
  CHECK(m == mem[1]);  // list 1's memory, rewritten on the same stream
  CHECK(f.count("alloc") == 0);
  CHECK(f.log.size() == 1 && f.log[0].kind == "upload" && f.log[0].mem == mem[1] &&
        f.log[0].stream == handle(1));
  f.log.clear();
  void* again = eager(c, f, 1);  // list 1 was evicted: uploaded anew
  CHECK(f.count("upload") == 1 && again != nullptr);
  CHECK(c.size() == 32);
}

void tables_last_used_on_another_stream_are_not_recycled() {
  Cache c;
  Fake f;
  std::vector<void*> mem;
  for (int id = 0; id < 32; ++id) mem.push_back(eager(c, f, id, 1));
  f.log.clear();
  void* other = eager(c, f, 500, 2);  // stream 2: no table of its own yet
  CHECK(f.count("alloc") == 1 && c.size() == 33);
  for (void* p : mem) CHECK(p != other);
  // list 5 moves to stream 2 (a later step, ordered after its stream-1 step)
  f.log.clear();
  CHECK(eager(c, f, 5, 2) == mem[5] && f.log.empty());
  // 30 more lists on stream 2 fill its share of 32; the next miss there recycles
  // stream 2's LRU (list 500), never a table whose latest use was stream 1
  for (int id = 600; id < 630; ++id) eager(c, f, id, 2);
  f.log.clear();
  void* r = eager(c, f, 700, 2);
  CHECK(r == other && f.count("alloc") == 0);
  // stream 1 now holds 31 tables; its next miss allocates (no recycling of
  // list 5, whose latest use was on stream 2)
  f.log.clear();
  void* s1 = eager(c, f, 800, 1);
  CHECK(f.count("alloc") == 1 && s1 != mem[5]);
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
  CHECK(c.acquire(f, 0, 1, t.data(), t.size(), true, handle(1), &mem, &slot) == madd_cache::kOk);
  c.release(slot);
  CHECK(mem == p && f.log.empty());  // nothing allocated or uploaded
  CHECK(c.pinned() == 1);
  for (int id = 200; id < 240; ++id) eager(c, f, id);
  CHECK(f.count("upload", p) == 0);
  f.log.clear();
  CHECK(eager(c, f, 7) == p);
  CHECK(f.count("upload") == 0);
  CHECK(c.size() == 33);  // 32 unpinned + the pinned one
}

void capture_miss_is_refused_without_side_effects() {
  Cache c;
  Fake f;
  eager(c, f, 1);
  f.log.clear();
  const std::vector<uint8_t> t = table(9);
  void* mem = nullptr;
  size_t slot = 0;
  CHECK(c.acquire(f, 0, 1, t.data(), t.size(), true, handle(1), &mem, &slot) ==
        madd_cache::kCaptureMiss);
  CHECK(f.log.empty() && mem == nullptr && c.size() == 1);
}

void a_list_longer_than_every_idle_table_gets_new_memory() {
  Cache c;
  Fake f;
  std::vector<void*> mem;
  for (int id = 0; id < 32; ++id) mem.push_back(eager(c, f, id, 1, 0, 3));
  f.log.clear();
  void* big = eager(c, f, 500, 1, 0, 300);  // 300 descriptors: more than a 64-descriptor table
  CHECK(f.count("alloc") == 1 && f.log.back().kind == "upload" && f.log.back().mem == big);
  for (void* p : mem) CHECK(p != big);
  // once present, a long table is recycled for a short list when it is the LRU
  for (int id = 0; id < 32; ++id) eager(c, f, id, 1, 0, 3);  // refresh the short ones
  f.log.clear();
  CHECK(eager(c, f, 900, 1, 0, 3) == big && f.count("alloc") == 0);
}

void held_tables_are_not_recycled() {
  Cache c;
  Fake f;
  std::vector<size_t> slots;
  for (int id = 0; id < 32; ++id) {
    const std::vector<uint8_t> t = table(id);
    void* mem = nullptr;
    size_t slot = 0;
    CHECK(c.acquire(f, 0, 1, t.data(), t.size(), false, handle(1), &mem, &slot) ==
          madd_cache::kOk);
    slots.push_back(slot);
  }
  f.log.clear();
  eager(c, f, 77);  // every table is held: the cache grows
  CHECK(f.count("alloc") == 1 && c.size() == 33);
  for (size_t s : slots) c.release(s);
}

void devices_are_separate() {
  Cache c;
  Fake f;
  for (int id = 0; id < 32; ++id) eager(c, f, id, 1, 0);
  f.log.clear();
  eager(c, f, 0, 1, 1);  // same bytes, other device: a miss there, no recycling here
  CHECK(f.count("alloc") == 1 && c.size() == 33);
  f.log.clear();
  eager(c, f, 0, 1, 0);  // still cached on device 0
  CHECK(f.count("upload") == 0);
}

void failed_allocation_leaves_a_usable_cache() {
  Cache c;
  Fake f;
  f.fail_alloc = true;
  const std::vector<uint8_t> t = table(3);
  void* mem = nullptr;
  size_t slot = 0;
  CHECK(c.acquire(f, 0, 1, t.data(), t.size(), false, handle(1), &mem, &slot) ==
        madd_cache::kNoMem);
  CHECK(c.size() == 0);
  f.fail_alloc = false;
  CHECK(eager(c, f, 3) != nullptr);
}

}  // namespace

int main() {
  hit_uploads_nothing();
  lru_of_the_same_stream_is_recycled_in_stream_order();
  tables_last_used_on_another_stream_are_not_recycled();
  pinned_table_survives_forty_lists();
  capture_miss_is_refused_without_side_effects();
  a_list_longer_than_every_idle_table_gets_new_memory();
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
