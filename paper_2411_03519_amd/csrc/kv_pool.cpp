// Host-side page pool and sequence table (see kv_pool.h).
#include "kv_pool.h"

#include <algorithm>
#include <functional>
#include <queue>
#include <unordered_set>

#include "../../include/metro.h"

namespace metro {

KvPagePool::KvPagePool(int32_t n_pages) : refcount_(n_pages, 0) {
  free_.reserve(n_pages);
  // lowest ids on top of the stack: pages are handed out in increasing order
  for (int32_t p = n_pages - 1; p >= 0; --p) free_.push_back(p);
}

bool KvPagePool::alloc(int32_t n, std::vector<int32_t>& out) {
  if (n < 0 || n > n_free()) return false;
  for (int32_t i = 0; i < n; ++i) {
    int32_t p = free_.back();
    free_.pop_back();
    refcount_[p] = 1;
    out.push_back(p);
  }
  return true;
}

void KvPagePool::ref(int32_t page) { ++refcount_.at(page); }

bool KvPagePool::unref(int32_t page) {
  if (page < 0 || page >= n_pages() || refcount_[page] <= 0) return false;
  if (--refcount_[page] == 0) free_.push_back(page);
  return true;
}

SequenceTable::SequenceTable(int32_t n_pages, int32_t page_size, int32_t max_seqs, int32_t max_context)
    : pool_(n_pages), page_size_(page_size), max_seqs_(max_seqs), max_context_(max_context) {}

int SequenceTable::open(int64_t* id) {
  if (open_count() >= max_seqs_) {
    err_ = "max_seqs sequences already open";
    return METRO_E_CAPACITY;
  }
  *id = next_id_++;
  Sequence s;
  s.hashable = cache_limit_ > 0;
  seqs_.emplace(*id, std::move(s));
  return METRO_OK;
}

int SequenceTable::open_cached(const int32_t* tokens, int32_t n, int64_t* id, int32_t* n_cached) {
  if (n < 0 || (n > 0 && !tokens)) {
    err_ = "open_cached: bad token list";
    return METRO_E_INVAL;
  }
  if (open_count() >= max_seqs_) {
    err_ = "max_seqs sequences already open";
    return METRO_E_CAPACITY;
  }
  Sequence s;
  s.hashable = cache_limit_ > 0;
  if (cache_limit_ > 0) {
    stats_.lookup_tokens += n;
    // walk the chain page by page; at least one token stays uncached
    Key k;
    k.parent = -1;
    for (int32_t i = 0; static_cast<int64_t>(i + 1) * page_size_ <= static_cast<int64_t>(n) - 1; ++i) {
      k.tokens.assign(tokens + static_cast<int64_t>(i) * page_size_, tokens + static_cast<int64_t>(i + 1) * page_size_);
      auto it = cache_.find(k);
      if (it == cache_.end()) break;
      s.pages.push_back(it->second);
      k.parent = it->second;
    }
    ++tick_;
    for (int32_t p : s.pages) {
      pool_.ref(p);
      entries_[p].last_use = tick_;
    }
    s.keyed = static_cast<int32_t>(s.pages.size());
    s.length = s.keyed * page_size_;
    s.chain = k.parent;
    stats_.hit_tokens += s.length;
  }
  *n_cached = s.length;
  *id = next_id_++;
  seqs_.emplace(*id, std::move(s));
  return METRO_OK;
}

const Sequence* SequenceTable::find(int64_t id) const {
  auto it = seqs_.find(id);
  return it == seqs_.end() ? nullptr : &it->second;
}

int SequenceTable::fork(int64_t src, int32_t n_tokens, int64_t* id, int32_t* copy_src, int32_t* copy_dst) {
  auto it = seqs_.find(src);
  if (it == seqs_.end()) {
    err_ = "fork: unknown sequence " + std::to_string(src);
    return METRO_E_SEQ;
  }
  const Sequence& s = it->second;
  if (n_tokens <= 0 || n_tokens > s.length) {
    err_ = "fork: n_tokens " + std::to_string(n_tokens) + " not in [1, " + std::to_string(s.length) + "]";
    return METRO_E_INVAL;
  }
  if (open_count() >= max_seqs_) {
    err_ = "max_seqs sequences already open";
    return METRO_E_CAPACITY;
  }
  const int32_t whole = n_tokens / page_size_;
  const bool partial = (n_tokens % page_size_) != 0;
  Sequence f;
  f.length = n_tokens;
  f.pages.assign(s.pages.begin(), s.pages.begin() + whole);
  *copy_src = *copy_dst = -1;
  if (partial) {
    std::vector<int32_t> fresh;
    if (!take_pages(1, fresh)) {
      err_ = "fork: no free page for the partial last page";
      return METRO_E_NOPAGES;
    }
    *copy_src = s.pages[whole];
    *copy_dst = fresh[0];
    f.pages.push_back(fresh[0]);
  }
  for (int32_t i = 0; i < whole; ++i) pool_.ref(f.pages[i]);
  *id = next_id_++;
  seqs_.emplace(*id, std::move(f));
  return METRO_OK;
}

int SequenceTable::close(int64_t id) {
  auto it = seqs_.find(id);
  if (it == seqs_.end()) {
    err_ = "close: unknown sequence " + std::to_string(id);
    return METRO_E_SEQ;
  }
  for (int32_t p : it->second.pages) pool_.unref(p);
  for (int32_t p : it->second.pins) pool_.unref(p);
  seqs_.erase(it);
  return METRO_OK;
}

int SequenceTable::reserve(const int64_t* ids, const int32_t* add, int32_t n) {
  std::unordered_set<int64_t> seen;
  int64_t need = 0;
  for (int32_t i = 0; i < n; ++i) {
    auto it = seqs_.find(ids[i]);
    if (it == seqs_.end()) {
      err_ = "unknown sequence " + std::to_string(ids[i]);
      return METRO_E_SEQ;
    }
    if (!seen.insert(ids[i]).second) {
      err_ = "sequence " + std::to_string(ids[i]) + " appears twice in one call";
      return METRO_E_INVAL;
    }
    if (add[i] < 0) {
      err_ = "negative token count";
      return METRO_E_INVAL;
    }
    const Sequence& s = it->second;
    const int64_t new_len = static_cast<int64_t>(s.length) + add[i];
    if (new_len > max_context_) {
      err_ = "sequence " + std::to_string(ids[i]) + " would hold " + std::to_string(new_len) +
             " tokens > max_context " + std::to_string(max_context_);
      return METRO_E_CAPACITY;
    }
    need += pages_for(static_cast<int32_t>(new_len)) - static_cast<int64_t>(s.pages.size());
  }
  if (need > pool_.n_free()) {
    const int64_t reclaim = cache_limit_ > 0 ? cache_only_pages() : 0;
    if (need > pool_.n_free() + reclaim) {
      err_ = "KV pool: call needs " + std::to_string(need) + " new pages, " + std::to_string(pool_.n_free()) +
             " free, " + std::to_string(reclaim) + " held only by the prefix cache";
      return METRO_E_NOPAGES;
    }
    evict(static_cast<int32_t>(need - pool_.n_free()));
    if (need > pool_.n_free()) {
      err_ = "KV pool: prefix cache could not release enough pages";
      return METRO_E_NOPAGES;
    }
  }
  for (int32_t i = 0; i < n; ++i) {
    Sequence& s = seqs_[ids[i]];
    const int32_t want = pages_for(s.length + add[i]) - static_cast<int32_t>(s.pages.size());
    if (want > 0) pool_.alloc(want, s.pages);
  }
  return METRO_OK;
}

void SequenceTable::commit(const int64_t* ids, const int32_t* add, int32_t n) {
  for (int32_t i = 0; i < n; ++i) seqs_[ids[i]].length += add[i];
}

// ---------------------------------------------------------------------------
// Prefix cache

size_t SequenceTable::KeyHash::operator()(const Key& k) const {
  // SplitMix64 finaliser over (parent, tokens...)
  auto mix = [](uint64_t z) {
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
  };
  uint64_t h = mix(static_cast<uint64_t>(static_cast<uint32_t>(k.parent)) + 0x9E3779B97F4A7C15ULL);
  for (int32_t t : k.tokens) h = mix(h ^ (static_cast<uint64_t>(static_cast<uint32_t>(t)) + 0x9E3779B97F4A7C15ULL));
  return static_cast<size_t>(h);
}

int32_t SequenceTable::cache_only_pages() const {
  int32_t n = 0;
  for (const auto& kv : entries_) n += pool_.refcount(kv.first) == 1;
  return n;
}

void SequenceTable::drop_entry(int32_t page) {
  auto it = entries_.find(page);
  if (it == entries_.end()) return;
  const int32_t parent = it->second.key.parent;
  if (parent >= 0) {
    auto pit = entries_.find(parent);
    if (pit != entries_.end()) --pit->second.children;
  }
  cache_.erase(it->second.key);
  entries_.erase(it);
  pool_.unref(page);
  ++stats_.evicted;
}

int32_t SequenceTable::evict(int32_t n) {
  // A sequence holding a cached page also holds every page of its prefix, so
  // the pages only the cache holds are closed under descendants: taking leaves
  // (no cached children) in least-recently-used order can reach all of them.
  using Item = std::pair<int64_t, int32_t>;  // (last use, page)
  std::priority_queue<Item, std::vector<Item>, std::greater<Item>> leaves;
  for (const auto& kv : entries_)
    if (kv.second.children == 0 && pool_.refcount(kv.first) == 1) leaves.emplace(kv.second.last_use, kv.first);
  int32_t dropped = 0;
  while (dropped < n && !leaves.empty()) {
    const int32_t page = leaves.top().second;
    leaves.pop();
    const int32_t parent = entries_.at(page).key.parent;
    drop_entry(page);
    ++dropped;
    if (parent >= 0) {
      auto pit = entries_.find(parent);
      if (pit != entries_.end() && pit->second.children == 0 && pool_.refcount(parent) == 1)
        leaves.emplace(pit->second.last_use, parent);
    }
  }
  return dropped;
}

bool SequenceTable::take_pages(int32_t n, std::vector<int32_t>& out) {
  if (n > pool_.n_free() && cache_limit_ > 0) {
    if (n > pool_.n_free() + cache_only_pages()) return false;
    evict(n - pool_.n_free());
  }
  return pool_.alloc(n, out);
}

void SequenceTable::enter_pages(Sequence& s) {
  while (s.hashable && static_cast<int32_t>(s.tail.size()) >= page_size_ &&
         s.keyed < static_cast<int32_t>(s.pages.size())) {
    Key k;
    k.parent = s.chain;
    k.tokens.assign(s.tail.begin(), s.tail.begin() + page_size_);
    const int32_t own = s.pages[s.keyed];
    auto it = cache_.find(k);
    if (it != cache_.end()) {
      // the same prefix is cached already (computed by another sequence):
      // keep that page alive as long as this sequence's chain names it
      const int32_t cp = it->second;
      if (cp != own) {
        pool_.ref(cp);
        s.pins.push_back(cp);
      }
      entries_.at(cp).last_use = ++tick_;
      s.chain = cp;
    } else {
      // the parent is held by this sequence, so eviction cannot take it
      if (static_cast<int32_t>(entries_.size()) >= cache_limit_ && evict(1) == 0) {
        s.hashable = false;
        break;
      }
      if (s.chain >= 0) ++entries_.at(s.chain).children;
      Entry e;
      e.key = k;
      e.last_use = ++tick_;
      cache_.emplace(std::move(k), own);
      entries_.emplace(own, std::move(e));
      pool_.ref(own);
      ++stats_.inserted;
      s.chain = own;
    }
    ++s.keyed;
    s.tail.erase(s.tail.begin(), s.tail.begin() + page_size_);
  }
  if (!s.hashable) s.tail.clear();
}

void SequenceTable::record_prefill(const int64_t* ids, const int32_t* cu, const int32_t* tokens, int32_t n) {
  if (cache_limit_ <= 0) return;
  for (int32_t i = 0; i < n; ++i) {
    auto it = seqs_.find(ids[i]);
    if (it == seqs_.end() || !it->second.hashable) continue;
    Sequence& s = it->second;
    s.tail.insert(s.tail.end(), tokens + cu[i], tokens + cu[i + 1]);
    if (static_cast<int64_t>(s.keyed) * page_size_ + static_cast<int64_t>(s.tail.size()) != s.length) {
      s.hashable = false;  // bookkeeping out of step: enter nothing more
      s.tail.clear();
      continue;
    }
    enter_pages(s);
  }
}

void SequenceTable::record_unknown(const int64_t* ids, int32_t n) {
  for (int32_t i = 0; i < n; ++i) {
    auto it = seqs_.find(ids[i]);
    if (it == seqs_.end()) continue;
    it->second.hashable = false;
    it->second.tail.clear();
  }
}

int SequenceTable::set_prefix_cache(int32_t max_pages) {
  if (max_pages < 0) {
    err_ = "prefix cache: negative page limit";
    return METRO_E_INVAL;
  }
  if (max_pages == 0) {
    for (auto& kv : seqs_) {
      kv.second.hashable = false;
      kv.second.chain = -1;
      kv.second.tail.clear();
    }
    for (const auto& kv : entries_) pool_.unref(kv.first);
    stats_.evicted += static_cast<int64_t>(entries_.size());
    entries_.clear();
    cache_.clear();
  } else if (static_cast<int32_t>(entries_.size()) > max_pages) {
    evict(static_cast<int32_t>(entries_.size()) - max_pages);
  }
  cache_limit_ = max_pages;
  return METRO_OK;
}

PrefixCacheStats SequenceTable::prefix_cache_stats() const {
  PrefixCacheStats st = stats_;
  st.pages = static_cast<int32_t>(entries_.size());
  st.limit = cache_limit_;
  return st;
}

}  // namespace metro
