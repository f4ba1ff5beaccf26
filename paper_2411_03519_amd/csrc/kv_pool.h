// Paged KV-cache bookkeeping on the host (no HIP dependency).
//
// The pool is a fixed set of pages; a page holds `page_size` consecutive
// positions of one sequence for every layer, K and V.  Sequences own an
// ordered block table of page ids.  Pages carry a reference count so that a
// forked sequence can share the whole pages of a common prompt prefix by
// reference (prefix sharing as in the serving engine of §4.1); a page is
// returned to the free stack when its last reference is dropped.
//
// Automatic prefix caching (the serving engine's common-prefix cache that the
// paper switches off for its measurements and credits with about 20% more
// throughput, §4.1): full pages whose tokens are all known on the host are
// entered in a cache keyed by (the cached page holding the previous 16
// positions, these 16 token ids).  The key therefore names the whole prefix up
// to and including the page, exactly -- two keys are equal only when the
// prefixes are equal token for token.  A new sequence opened with its prompt
// attaches the longest chain of cached pages that matches the prompt.  The
// cache holds one reference per cached page; pages only the cache holds are
// evicted least recently used first, leaves before their parents, when the
// pool runs dry or the cache reaches its page limit.
//
// Every mutating operation is all-or-nothing: on failure nothing changes
// (evicting pages that only the cache holds aside, which changes no sequence).
#pragma once

#include <cstdint>
#include <string>
#include <unordered_map>
#include <vector>

namespace metro {

class KvPagePool {
 public:
  explicit KvPagePool(int32_t n_pages);

  int32_t n_pages() const { return static_cast<int32_t>(refcount_.size()); }
  int32_t n_free() const { return static_cast<int32_t>(free_.size()); }
  int32_t refcount(int32_t page) const { return refcount_.at(page); }

  // Take n pages (refcount 1) and append them to `out`; false (and no change)
  // when fewer than n pages are free.
  bool alloc(int32_t n, std::vector<int32_t>& out);
  // Add a reference to a page in use.
  void ref(int32_t page);
  // Drop a reference; the page becomes free at zero.  Returns false for a page
  // that is not in use (double free) without changing anything.
  bool unref(int32_t page);

 private:
  std::vector<int32_t> free_;      // stack of free page ids
  std::vector<int32_t> refcount_;  // per page
};

struct Sequence {
  int32_t length = 0;             // tokens written
  std::vector<int32_t> pages;     // block table
  // prefix-cache bookkeeping
  bool hashable = false;          // every token so far is known on the host
  int32_t keyed = 0;              // leading pages already entered or matched
  int32_t chain = -1;             // cached page holding the last keyed page's prefix (-1: none yet)
  std::vector<int32_t> tail;      // known tokens past the keyed pages
  std::vector<int32_t> pins;      // extra references to cached pages equal to own pages
};

struct PrefixCacheStats {
  int32_t pages = 0;              // pages the cache holds
  int32_t limit = 0;              // 0 = caching off
  int64_t lookup_tokens = 0;      // prompt tokens offered to open_cached
  int64_t hit_tokens = 0;         // of which attached from the cache
  int64_t inserted = 0;           // pages entered
  int64_t evicted = 0;            // pages dropped
};

// Sequences of one model: handles, lengths, block tables.
class SequenceTable {
 public:
  SequenceTable(int32_t n_pages, int32_t page_size, int32_t max_seqs, int32_t max_context);

  KvPagePool& pool() { return pool_; }
  const KvPagePool& pool() const { return pool_; }
  int32_t page_size() const { return page_size_; }
  int32_t open_count() const { return static_cast<int32_t>(seqs_.size()); }

  // Returns 0 or a metro_status code (negative).
  int open(int64_t* id);
  // Open a sequence and attach the longest chain of cached pages matching
  // tokens[0 .. n), at most n - 1 tokens (so at least one is left to run);
  // *n_cached = the tokens attached (a multiple of the page size, 0 when
  // caching is off).
  int open_cached(const int32_t* tokens, int32_t n, int64_t* id, int32_t* n_cached);
  // Fork: the new sequence shares src's whole pages covering [0, n_tokens);
  // when n_tokens is not a page multiple a fresh page is taken for the partial
  // last page and *copy_src / *copy_dst name the page to copy (else -1).
  int fork(int64_t src, int32_t n_tokens, int64_t* id, int32_t* copy_src, int32_t* copy_dst);
  int close(int64_t id);
  const Sequence* find(int64_t id) const;

  // Reserve pages so that each sequence ids[i] can grow by add[i] tokens.
  // All-or-nothing over the whole list (E_NOPAGES, E_CAPACITY, E_SEQ, E_INVAL
  // for a repeated id).  On success the block tables are extended but lengths
  // are unchanged; call commit() once the work has been enqueued.
  int reserve(const int64_t* ids, const int32_t* add, int32_t n);
  void commit(const int64_t* ids, const int32_t* add, int32_t n);

  // After a committed prefill: items ids[i] received tokens[cu[i] .. cu[i+1]);
  // their newly filled pages are entered in the cache.
  void record_prefill(const int64_t* ids, const int32_t* cu, const int32_t* tokens, int32_t n);
  // After a committed decode step: the new tokens are not known on the host,
  // so these sequences enter no further pages.
  void record_unknown(const int64_t* ids, int32_t n);

  // Turn caching on with a limit of max_pages cached pages, or off (0), which
  // drops every cached page and stops every open sequence from entering more.
  int set_prefix_cache(int32_t max_pages);
  PrefixCacheStats prefix_cache_stats() const;
  // Pages only the cache holds (evictable).
  int32_t cache_only_pages() const;
  bool cached(int32_t page) const { return entries_.count(page) != 0; }

  const std::string& error() const { return err_; }

 private:
  int32_t pages_for(int32_t tokens) const { return (tokens + page_size_ - 1) / page_size_; }

  struct Key {
    int32_t parent;
    std::vector<int32_t> tokens;
    bool operator==(const Key& o) const { return parent == o.parent && tokens == o.tokens; }
  };
  struct KeyHash {
    size_t operator()(const Key& k) const;
  };
  struct Entry {
    Key key;
    int32_t children = 0;         // cached pages whose key names this page
    int64_t last_use = 0;
  };
  // Drop up to n pages only the cache holds, least recently used leaves first;
  // returns the number dropped.
  int32_t evict(int32_t n);
  void drop_entry(int32_t page);
  void enter_pages(Sequence& s);
  // alloc() that first evicts pages only the cache holds when too few are
  // free; false (nothing changed) when that still is not enough.
  bool take_pages(int32_t n, std::vector<int32_t>& out);

  std::unordered_map<Key, int32_t, KeyHash> cache_;     // key -> page
  std::unordered_map<int32_t, Entry> entries_;          // page -> entry
  int32_t cache_limit_ = 0;
  int64_t tick_ = 0;
  PrefixCacheStats stats_;

  KvPagePool pool_;
  int32_t page_size_;
  int32_t max_seqs_;
  int32_t max_context_;
  int64_t next_id_ = 1;
  std::unordered_map<int64_t, Sequence> seqs_;
  std::string err_;
};

}  // namespace metro
