// Host-only unit test of the KV page pool and sequence table (built with g++).
#include <cassert>
#include <cstdio>
#include <set>
#include <vector>

#include "../include/metro.h"
#include "../paper_2411_03519_amd/csrc/kv_pool.h"

using metro::SequenceTable;

#define CHECK(c)                                                   \
  do {                                                             \
    if (!(c)) {                                                    \
      std::fprintf(stderr, "FAIL %s:%d: %s\n", __FILE__, __LINE__, #c); \
      return 1;                                                    \
    }                                                              \
  } while (0)

int main() {
  // pool basics
  {
    metro::KvPagePool p(4);
    std::vector<int32_t> got;
    CHECK(p.alloc(3, got) && got.size() == 3 && p.n_free() == 1);
    CHECK(got[0] == 0 && got[1] == 1 && got[2] == 2);
    CHECK(!p.alloc(2, got) && got.size() == 3 && p.n_free() == 1);  // all-or-nothing
    p.ref(1);
    CHECK(p.refcount(1) == 2);
    CHECK(p.unref(1) && p.n_free() == 1);
    CHECK(p.unref(1) && p.n_free() == 2);
    CHECK(!p.unref(1) && p.n_free() == 2);  // double free refused
    CHECK(!p.unref(99));
  }
  // sequences: reserve / commit / exhaustion
  {
    SequenceTable t(10, 16, 3, 150);
    int64_t a, b, c, d;
    CHECK(t.open(&a) == METRO_OK && t.open(&b) == METRO_OK && t.open(&c) == METRO_OK);
    CHECK(t.open(&d) == METRO_E_CAPACITY);
    int64_t ids[2] = {a, b};
    int32_t add[2] = {100, 0};
    CHECK(t.reserve(ids, add, 2) == METRO_OK);
    CHECK(t.find(a)->pages.size() == 7 && t.find(a)->length == 0);
    t.commit(ids, add, 2);
    CHECK(t.find(a)->length == 100 && t.pool().n_free() == 3);
    int32_t add2[2] = {13, 40};  // 1 + 3 pages, 3 free
    CHECK(t.reserve(ids, add2, 2) == METRO_E_NOPAGES);
    CHECK(t.find(a)->pages.size() == 7 && t.find(b)->pages.empty() && t.pool().n_free() == 3);
    int64_t dup[2] = {a, a};
    int32_t one[2] = {1, 1};
    CHECK(t.reserve(dup, one, 2) == METRO_E_INVAL);
    int64_t unk[1] = {999};
    CHECK(t.reserve(unk, one, 1) == METRO_E_SEQ);
    int32_t big[1] = {51};
    CHECK(t.reserve(ids, big, 1) == METRO_E_CAPACITY);  // 151 > max_context
    CHECK(t.pool().n_free() == 3);
    // fork at a page boundary: all pages shared
    int64_t f;
    int32_t cs, cd;
    CHECK(t.close(c) == METRO_OK);
    CHECK(t.fork(a, 96, &f, &cs, &cd) == METRO_OK && cs == -1 && cd == -1);
    CHECK(t.find(f)->pages.size() == 6 && t.find(f)->length == 96);
    for (int i = 0; i < 6; ++i) CHECK(t.pool().refcount(t.find(a)->pages[i]) == 2);
    CHECK(t.pool().refcount(t.find(a)->pages[6]) == 1);
    // closing the source keeps the shared pages alive
    CHECK(t.close(a) == METRO_OK);
    CHECK(t.pool().n_free() == 4);
    for (int32_t pg : t.find(f)->pages) CHECK(t.pool().refcount(pg) == 1);
    // fork inside a page: a fresh page for the copied tail
    int64_t g;
    CHECK(t.fork(f, 40, &g, &cs, &cd) == METRO_OK);
    CHECK(cs == t.find(f)->pages[2] && cd == t.find(g)->pages[2] && cs != cd);
    CHECK(t.find(g)->pages.size() == 3 && t.pool().n_free() == 3);
    CHECK(t.fork(f, 97, &g, &cs, &cd) == METRO_E_INVAL);
    CHECK(t.fork(f, 0, &g, &cs, &cd) == METRO_E_INVAL);
    CHECK(t.fork(12345, 1, &g, &cs, &cd) == METRO_E_SEQ);
    CHECK(t.close(f) == METRO_OK && t.close(g) == METRO_OK);
    CHECK(t.pool().n_free() == 10);
    CHECK(t.close(g) == METRO_E_SEQ);
  }
  // randomised: refcounts always equal the number of block-table entries
  {
    SequenceTable t(64, 16, 32, 400);
    std::vector<int64_t> open;
    unsigned s = 12345;
    auto rnd = [&](unsigned n) { s = s * 1103515245u + 12345u; return (s >> 8) % n; };
    for (int it = 0; it < 4000; ++it) {
      const unsigned op = rnd(4);
      int32_t cs, cd;
      if (op == 0 || open.empty()) {
        int64_t id;
        if (t.open(&id) == METRO_OK) open.push_back(id);
      } else if (op == 1) {
        const size_t k = rnd(open.size());
        t.close(open[k]);
        open.erase(open.begin() + k);
      } else if (op == 2) {
        int64_t id = open[rnd(open.size())];
        int32_t n = static_cast<int32_t>(1 + rnd(40));
        if (t.reserve(&id, &n, 1) == METRO_OK) t.commit(&id, &n, 1);
      } else {
        int64_t src = open[rnd(open.size())], id;
        const int32_t len = t.find(src)->length;
        if (len > 0 && t.fork(src, static_cast<int32_t>(1 + rnd(len)), &id, &cs, &cd) == METRO_OK) open.push_back(id);
      }
      std::vector<int> cnt(64, 0);
      for (int64_t id : open) {
        const metro::Sequence* q = t.find(id);
        CHECK(static_cast<int>(q->pages.size()) == (q->length + 15) / 16);
        for (int32_t pg : q->pages) ++cnt[pg];
      }
      int used = 0;
      for (int pg = 0; pg < 64; ++pg) {
        CHECK(cnt[pg] == t.pool().refcount(pg));
        used += cnt[pg] > 0;
      }
      CHECK(used + t.pool().n_free() == 64);
    }
  }
  std::printf("kvpool ok\n");
  return 0;
}
