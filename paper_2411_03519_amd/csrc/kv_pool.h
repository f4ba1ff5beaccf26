// Paged KV-cache bookkeeping on the host (no HIP dependency).
//
// The pool is a fixed set of pages; a page holds `page_size` consecutive
// positions of one sequence for every layer, K and V.  Sequences own an
// ordered block table of page ids.  Pages carry a reference count so that a
// forked sequence can share the whole pages of a common prompt prefix by
// reference (prefix sharing as in the serving engine of §4.1); a page is
// returned to the free stack when its last reference is dropped.
//
// Every mutating operation is all-or-nothing: on failure nothing changes.
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

  const std::string& error() const { return err_; }

 private:
  int32_t pages_for(int32_t tokens) const { return (tokens + page_size_ - 1) / page_size_; }

  KvPagePool pool_;
  int32_t page_size_;
  int32_t max_seqs_;
  int32_t max_context_;
  int64_t next_id_ = 1;
  std::unordered_map<int64_t, Sequence> seqs_;
  std::string err_;
};

}  // namespace metro
