// Host-side page pool and sequence table (see kv_pool.h).
#include "kv_pool.h"

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
  seqs_.emplace(*id, Sequence{});
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
    if (!pool_.alloc(1, fresh)) {
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
    err_ = "KV pool: call needs " + std::to_string(need) + " new pages, " + std::to_string(pool_.n_free()) +
           " free";
    return METRO_E_NOPAGES;
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

}  // namespace metro
