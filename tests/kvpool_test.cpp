// Host-only unit test of the KV page pool and sequence table (built with g++).
#include <algorithm>
#include <cassert>
#include <cstdio>
#include <cstring>
#include <iostream>
#include <map>
#include <set>
#include <string>
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

// reserve + commit + record_prefill of n known tokens on one sequence
static int prefill(SequenceTable& t, int64_t id, const int32_t* tok, int32_t n) {
  const int r = t.reserve(&id, &n, 1);
  if (r != METRO_OK) return r;
  t.commit(&id, &n, 1);
  const int32_t cu[2] = {0, n};
  t.record_prefill(&id, cu, tok, 1);
  return METRO_OK;
}

static std::vector<int32_t> pages_of(const SequenceTable& t, int64_t id) { return t.find(id)->pages; }

static int prefix_cache_tests() {
  // entering pages, lookups, the at-most-n-1 rule, chain identity
  {
    SequenceTable t(20, 16, 8, 400);
    CHECK(t.set_prefix_cache(100) == METRO_OK);
    std::vector<int32_t> A(70);
    for (int i = 0; i < 70; ++i) A[i] = 1000 + i;
    int64_t a;
    CHECK(t.open(&a) == METRO_OK && t.find(a)->hashable);
    CHECK(prefill(t, a, A.data(), 40) == METRO_OK);
    CHECK(t.prefix_cache_stats().pages == 2 && t.find(a)->keyed == 2 && t.find(a)->tail.size() == 8);
    const std::vector<int32_t> pa0 = pages_of(t, a);
    CHECK(t.cached(pa0[0]) && t.cached(pa0[1]) && !t.cached(pa0[2]));
    CHECK(t.pool().refcount(pa0[0]) == 2 && t.pool().refcount(pa0[2]) == 1);
    CHECK(prefill(t, a, A.data() + 40, 30) == METRO_OK);
    CHECK(t.prefix_cache_stats().pages == 4 && t.find(a)->tail.size() == 6);
    const std::vector<int32_t> pa = pages_of(t, a);
    int64_t b;
    int32_t nc = -1;
    CHECK(t.open_cached(A.data(), 70, &b, &nc) == METRO_OK && nc == 64);
    CHECK(t.find(b)->length == 64 && t.find(b)->keyed == 4);
    for (int i = 0; i < 4; ++i) CHECK(t.find(b)->pages[i] == pa[i] && t.pool().refcount(pa[i]) == 3);
    CHECK(t.close(b) == METRO_OK);
    CHECK(t.open_cached(A.data(), 64, &b, &nc) == METRO_OK && nc == 48 && t.close(b) == METRO_OK);
    CHECK(t.open_cached(A.data(), 65, &b, &nc) == METRO_OK && nc == 64 && t.close(b) == METRO_OK);
    CHECK(t.open_cached(A.data(), 16, &b, &nc) == METRO_OK && nc == 0 && t.close(b) == METRO_OK);
    CHECK(t.open_cached(A.data(), 17, &b, &nc) == METRO_OK && nc == 16 && t.close(b) == METRO_OK);
    CHECK(t.open_cached(nullptr, 0, &b, &nc) == METRO_OK && nc == 0 && t.close(b) == METRO_OK);
    CHECK(t.open_cached(nullptr, 5, &b, &nc) == METRO_E_INVAL);
    // a page is found only under its whole prefix
    std::vector<int32_t> B = A;
    B[0] = 7;
    CHECK(t.open_cached(B.data(), 70, &b, &nc) == METRO_OK && nc == 0 && t.close(b) == METRO_OK);
    B = A;
    B[20] = 7;
    CHECK(t.open_cached(B.data(), 70, &b, &nc) == METRO_OK && nc == 16 && t.close(b) == METRO_OK);
    const metro::PrefixCacheStats st = t.prefix_cache_stats();
    CHECK(st.inserted == 4 && st.evicted == 0 && st.limit == 100);
    CHECK(st.hit_tokens == 64 + 48 + 64 + 16 + 16 && st.lookup_tokens == 70 + 64 + 65 + 16 + 17 + 70 + 70);

    // the same prefix computed again by another sequence: its pages are not
    // entered, the cached ones are pinned, and its chain continues from them
    std::vector<int32_t> C(A.begin(), A.begin() + 48);
    for (int i = 0; i < 26; ++i) C.push_back(5000 + i);
    int64_t c;
    CHECK(t.open(&c) == METRO_OK && prefill(t, c, C.data(), 74) == METRO_OK);
    CHECK(t.prefix_cache_stats().pages == 5 && t.find(c)->pins.size() == 3);
    const std::vector<int32_t> pc = pages_of(t, c);
    CHECK(!t.cached(pc[0]) && t.cached(pc[3]) && t.pool().refcount(pa[0]) == 3);
    CHECK(t.open_cached(C.data(), 74, &b, &nc) == METRO_OK && nc == 64);
    CHECK(t.find(b)->pages[0] == pa[0] && t.find(b)->pages[2] == pa[2] && t.find(b)->pages[3] == pc[3]);
    CHECK(t.close(b) == METRO_OK);
    // unknown (decoded) tokens end the sequence's entries
    int32_t one = 1;
    CHECK(t.reserve(&c, &one, 1) == METRO_OK);
    t.commit(&c, &one, 1);
    t.record_unknown(&c, 1);
    CHECK(!t.find(c)->hashable && t.find(c)->tail.empty());
    CHECK(prefill(t, c, C.data(), 30) == METRO_OK && t.prefix_cache_stats().pages == 5);
    // closing drops the pins; turning the cache off frees every cached page
    CHECK(t.close(c) == METRO_OK && t.close(a) == METRO_OK);
    CHECK(t.cache_only_pages() == 5 && t.pool().n_free() == 15);
    CHECK(t.set_prefix_cache(0) == METRO_OK && t.pool().n_free() == 20 && t.prefix_cache_stats().pages == 0);
    CHECK(t.open_cached(A.data(), 70, &b, &nc) == METRO_OK && nc == 0 && !t.find(b)->hashable);
    CHECK(t.set_prefix_cache(-1) == METRO_E_INVAL);
  }
  // eviction: least recently used leaves first, only pages no sequence holds,
  // and a call that cannot be served evicts nothing
  {
    SequenceTable t(8, 16, 8, 400);
    CHECK(t.set_prefix_cache(100) == METRO_OK);
    std::vector<int32_t> A(64), B(96);
    for (int i = 0; i < 64; ++i) A[i] = i;
    for (int i = 0; i < 96; ++i) B[i] = 500 + i;
    int64_t a, b, c;
    CHECK(t.open(&a) == METRO_OK && prefill(t, a, A.data(), 64) == METRO_OK);
    const std::vector<int32_t> pa = pages_of(t, a);
    CHECK(t.close(a) == METRO_OK && t.pool().n_free() == 4 && t.cache_only_pages() == 4);
    CHECK(t.open(&b) == METRO_OK);
    int32_t n9 = 144;  // 9 pages > 4 free + 4 cached
    CHECK(t.reserve(&b, &n9, 1) == METRO_E_NOPAGES && t.prefix_cache_stats().pages == 4);
    CHECK(prefill(t, b, B.data(), 96) == METRO_OK);  // 6 pages: 2 evicted, the deepest two
    CHECK(t.prefix_cache_stats().evicted == 2 && t.cached(pa[0]) && t.cached(pa[1]));
    const std::vector<int32_t> pb = pages_of(t, b);
    CHECK(std::count(pb.begin(), pb.end(), pa[2]) == 1 && std::count(pb.begin(), pb.end(), pa[3]) == 1);
    CHECK(t.prefix_cache_stats().pages == 8);
    int32_t nc;
    CHECK(t.open_cached(A.data(), 64, &c, &nc) == METRO_OK && nc == 32);
    CHECK(t.close(b) == METRO_OK && t.close(c) == METRO_OK);
    CHECK(t.pool().n_free() == 0 && t.cache_only_pages() == 8);
    // a lower limit evicts down to it: b's five deepest pages (A's two were
    // used more recently)
    CHECK(t.set_prefix_cache(3) == METRO_OK && t.prefix_cache_stats().pages == 3);
    CHECK(t.cached(pa[0]) && t.cached(pa[1]) && t.cached(pb[0]) && !t.cached(pb[1]));
    // at the limit, entering a page evicts one only the cache holds; once none
    // is left the sequence stops entering pages
    CHECK(t.open(&a) == METRO_OK && prefill(t, a, B.data(), 96) == METRO_OK);
    CHECK(t.prefix_cache_stats().pages == 3 && !t.find(a)->hashable);
    CHECK(!t.cached(pa[0]) && !t.cached(pa[1]));
    CHECK(t.open_cached(B.data(), 96, &c, &nc) == METRO_OK && nc == 48 && t.close(c) == METRO_OK);
    CHECK(t.close(a) == METRO_OK);
  }
  return 0;
}

// Randomised prefix-cache run: refcounts equal block-table entries + pins +
// cache entries; every full page of every sequence holds exactly that
// sequence's prefix (the tokens from position 0 through the page's end).
static int prefix_cache_random() {
  const int NP = 48;
  SequenceTable t(NP, 16, 12, 300);
  CHECK(t.set_prefix_cache(40) == METRO_OK);
  unsigned s = 777;
  auto rnd = [&](unsigned n) { s = s * 1103515245u + 12345u; return (s >> 8) % n; };
  std::map<int64_t, std::vector<int32_t>> toks;   // every sequence's tokens
  std::map<int32_t, std::vector<int32_t>> written;  // page -> prefix its K/V was computed from
  auto make_prompt = [&]() {
    std::vector<int32_t> p;
    const int fam = static_cast<int>(rnd(3));
    const int shared = static_cast<int>(rnd(80));
    for (int i = 0; i < shared; ++i) p.push_back(fam * 100 + i % 7);
    const int own = 1 + static_cast<int>(rnd(50));
    for (int i = 0; i < own; ++i) p.push_back(static_cast<int32_t>(rnd(4)));
    return p;
  };
  auto note_written = [&](int64_t id, int32_t from) {
    const metro::Sequence* q = t.find(id);
    const std::vector<int32_t>& tk = toks[id];
    for (int32_t pg = from / 16; pg < static_cast<int32_t>(q->pages.size()); ++pg) {
      const int32_t end = std::min<int32_t>(q->length, 16 * (pg + 1));
      written[q->pages[pg]] = std::vector<int32_t>(tk.begin(), tk.begin() + end);
    }
  };
  for (int it = 0; it < 6000; ++it) {
    const unsigned op = rnd(7);
    if (toks.empty() || op == 0) {
      std::vector<int32_t> p = make_prompt();
      int64_t id;
      int32_t nc;
      if (t.open_cached(p.data(), static_cast<int32_t>(p.size()), &id, &nc) != METRO_OK) continue;
      CHECK(nc % 16 == 0 && nc < static_cast<int32_t>(p.size()));
      toks[id] = std::vector<int32_t>(p.begin(), p.begin() + nc);
      const int32_t rest = static_cast<int32_t>(p.size()) - nc;
      if (prefill(t, id, p.data() + nc, rest) == METRO_OK) {
        toks[id] = p;
        note_written(id, nc);
      }
    } else if (op == 1) {
      auto itq = toks.begin();
      std::advance(itq, rnd(toks.size()));
      CHECK(t.close(itq->first) == METRO_OK);
      toks.erase(itq);
    } else if (op == 2 || op == 3) {
      auto itq = toks.begin();
      std::advance(itq, rnd(toks.size()));
      const int64_t id = itq->first;
      std::vector<int32_t> more;
      const int n = 1 + static_cast<int>(rnd(30));
      for (int i = 0; i < n; ++i) more.push_back(static_cast<int32_t>(rnd(4)));
      const int32_t from = t.find(id)->length;
      if (op == 2) {
        if (prefill(t, id, more.data(), n) != METRO_OK) continue;
      } else {
        int32_t one = 1;
        more.resize(1);
        if (t.reserve(&id, &one, 1) != METRO_OK) continue;
        t.commit(&id, &one, 1);
        t.record_unknown(&id, 1);
      }
      toks[id].insert(toks[id].end(), more.begin(), more.end());
      note_written(id, from);
    } else if (op == 4) {
      auto itq = toks.begin();
      std::advance(itq, rnd(toks.size()));
      const int32_t len = t.find(itq->first)->length;
      int64_t id;
      int32_t cs, cd;
      if (len > 0) {
        const int32_t n = 1 + static_cast<int32_t>(rnd(len));
        if (t.fork(itq->first, n, &id, &cs, &cd) == METRO_OK) {
          toks[id] = std::vector<int32_t>(itq->second.begin(), itq->second.begin() + n);
          if (cd >= 0) written[cd] = std::vector<int32_t>(toks[id].begin(), toks[id].end());
        }
      }
    } else if (op == 5 && rnd(40) == 0) {
      CHECK(t.set_prefix_cache(rnd(3) == 0 ? 0 : 10 + static_cast<int32_t>(rnd(40))) == METRO_OK);
    }
    // invariants
    std::vector<int> cnt(NP, 0);
    for (const auto& kv : toks) {
      const metro::Sequence* q = t.find(kv.first);
      CHECK(q && q->length == static_cast<int32_t>(kv.second.size()));
      CHECK(static_cast<int>(q->pages.size()) == (q->length + 15) / 16);
      for (size_t pg = 0; pg < q->pages.size(); ++pg) {
        ++cnt[q->pages[pg]];
        const int32_t end = std::min<int32_t>(q->length, 16 * static_cast<int32_t>(pg + 1));
        const std::vector<int32_t>& w = written[q->pages[pg]];
        CHECK(static_cast<int32_t>(w.size()) >= end);
        CHECK(std::equal(kv.second.begin(), kv.second.begin() + end, w.begin()));
      }
      for (int32_t pg : q->pins) ++cnt[pg];
    }
    int used = 0;
    for (int pg = 0; pg < NP; ++pg) {
      CHECK(cnt[pg] + (t.cached(pg) ? 1 : 0) == t.pool().refcount(pg));
      used += t.pool().refcount(pg) > 0;
    }
    CHECK(used + t.pool().n_free() == NP);
    CHECK(t.prefix_cache_stats().pages <= std::max(t.prefix_cache_stats().limit, 40));
  }
  const metro::PrefixCacheStats st = t.prefix_cache_stats();
  CHECK(st.hit_tokens > 0 && st.evicted > 0 && st.inserted > 0);
  std::printf("prefix cache random: %lld lookup tokens, %lld hits, %lld entered, %lld evicted\n",
              (long long)st.lookup_tokens, (long long)st.hit_tokens, (long long)st.inserted, (long long)st.evicted);
  return 0;
}

// Replay a script of sequence operations from stdin (one per line, ids are
// the script's own):
//   o ID                open            c ID N t1..tN    open_cached
//   p ID N t1..tN       prefill         d ID             decode one token
//   f ID SRC N          fork            x ID             close
// and print "c ID n_cached" for every open_cached, in order.  The pool is
// large and the cache limit high, so nothing is evicted.
static int replay() {
  SequenceTable t(1 << 14, 16, 1 << 12, 1 << 14);
  if (t.set_prefix_cache(1 << 14) != METRO_OK) return 1;
  std::map<long long, int64_t> ids;
  std::string op;
  while (std::cin >> op) {
    long long id;
    std::cin >> id;
    if (op == "o") {
      int64_t h;
      if (t.open(&h) != METRO_OK) return 2;
      ids[id] = h;
    } else if (op == "c" || op == "p") {
      int32_t n;
      std::cin >> n;
      std::vector<int32_t> tok(n);
      for (auto& v : tok) std::cin >> v;
      if (op == "c") {
        int64_t h;
        int32_t nc;
        if (t.open_cached(tok.data(), n, &h, &nc) != METRO_OK) return 3;
        ids[id] = h;
        std::printf("c %lld %d\n", id, nc);
      } else if (prefill(t, ids.at(id), tok.data(), n) != METRO_OK) {
        return 4;
      }
    } else if (op == "d") {
      int64_t h = ids.at(id);
      int32_t one = 1;
      if (t.reserve(&h, &one, 1) != METRO_OK) return 5;
      t.commit(&h, &one, 1);
      t.record_unknown(&h, 1);
    } else if (op == "f") {
      long long src;
      int32_t n, cs, cd;
      std::cin >> src >> n;
      int64_t h;
      if (t.fork(ids.at(src), n, &h, &cs, &cd) != METRO_OK) return 6;
      ids[id] = h;
    } else if (op == "x") {
      if (t.close(ids.at(id)) != METRO_OK) return 7;
      ids.erase(id);
    } else {
      return 8;
    }
  }
  return 0;
}

int main(int argc, char** argv) {
  if (argc > 1 && std::strcmp(argv[1], "replay") == 0) return replay();
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
  if (prefix_cache_tests() != 0 || prefix_cache_random() != 0) return 1;
  std::printf("kvpool ok\n");
  return 0;
}
