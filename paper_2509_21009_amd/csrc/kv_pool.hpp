// Paged KV-cache page pool (host side).
//
// Long-tailed response lengths (paper section 2.2) make reserving the
// maximum length per sequence wasteful; the KV cache is instead split into
// fixed-size pages that are handed to a sequence as its context grows and
// returned when it finishes, so memory follows the live, shrinking batch
// (section 4.2 discusses the KV pressure that otherwise causes preemption).
// Admission checks the projected need against the free pages first (the
// projection of historical lengths x per-token KV footprint in section 4.4,
// exact here because response lengths are given).
//
// This class only manages page ids; the device page table and the KV bytes
// live in the engine.  It is plain host C++ so it is testable without a GPU.
#pragma once

#include <cstdint>
#include <stdexcept>
#include <vector>

namespace rollpack {

class PagePool {
 public:
  explicit PagePool(int64_t n_pages) : n_pages_(n_pages), owner_(n_pages, -1) {
    free_.reserve(static_cast<size_t>(n_pages));
    // Hand out low page ids first: pop from the back of a descending list.
    for (int64_t p = n_pages - 1; p >= 0; --p) free_.push_back(static_cast<int32_t>(p));
  }

  int64_t capacity() const { return n_pages_; }
  int64_t free_pages() const { return static_cast<int64_t>(free_.size()); }
  int64_t used_pages() const { return n_pages_ - free_pages(); }
  int64_t peak_used() const { return peak_; }
  void reset_peak() { peak_ = used_pages(); }

  static int64_t pages_for(int64_t tokens, int32_t page_tokens) {
    return tokens <= 0 ? 0 : (tokens + page_tokens - 1) / page_tokens;
  }

  // True if `pages` more pages can be taken now.
  bool can_take(int64_t pages) const { return pages <= free_pages(); }

  // Take `count` pages for `owner` (an opaque non-negative id), appending
  // them to `out`.  Throws std::runtime_error without side effects when the
  // pool is short.
  void take(int64_t count, int64_t owner, std::vector<int32_t>& out) {
    if (owner < 0) throw std::invalid_argument("page owner must be non-negative");
    if (count < 0 || count > free_pages()) throw std::runtime_error("out of KV pages");
    out.reserve(out.size() + static_cast<size_t>(count));
    for (int64_t i = 0; i < count; ++i) {
      int32_t p = free_.back();
      free_.pop_back();
      owner_[p] = owner;
      out.push_back(p);
    }
    if (used_pages() > peak_) peak_ = used_pages();
  }

  // Return pages previously taken by `owner`.  Every page must be owned by it.
  void give_back(const std::vector<int32_t>& pages, int64_t owner) {
    for (int32_t p : pages) {
      if (p < 0 || p >= n_pages_ || owner_[p] != owner)
        throw std::logic_error("page returned by a sequence that does not own it");
    }
    for (int32_t p : pages) {
      owner_[p] = -1;
      free_.push_back(p);
    }
  }

  int64_t owner_of(int32_t page) const { return owner_.at(static_cast<size_t>(page)); }

 private:
  int64_t n_pages_;
  int64_t peak_ = 0;
  std::vector<int32_t> free_;
  std::vector<int64_t> owner_;
};

}  // namespace rollpack
