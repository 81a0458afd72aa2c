// Host page allocator of the paged KV cache.  Pure C++ (no HIP) so that it can
// be tested on a machine without a GPU.
//
// Page indices are a deterministic function of the history of lengths:
// allocation always takes the lowest-numbered free page, and a page returns
// to the pool as soon as it holds no position below its sequence's length.
#pragma once

#include <cstdint>
#include <functional>
#include <queue>
#include <vector>

namespace spec {

class PagePool {
 public:
  explicit PagePool(int num_pages = 0, int page_size = 16) { reset(num_pages, page_size); }

  void reset(int num_pages, int page_size) {
    page_size_ = page_size;
    num_pages_ = num_pages;
    free_ = decltype(free_)();
    for (int p = 0; p < num_pages; ++p) free_.push(p);
  }

  int page_size() const { return page_size_; }
  int num_pages() const { return num_pages_; }
  int free_pages() const { return static_cast<int>(free_.size()); }
  int pages_for(int64_t length) const {
    return static_cast<int>((length + page_size_ - 1) / page_size_);
  }
  // pages a table must gain to cover positions 0..length-1
  int need(const std::vector<int32_t>& table, int64_t length) const {
    const int n = pages_for(length) - static_cast<int>(table.size());
    return n > 0 ? n : 0;
  }
  // Extend `table` to cover 0..length-1; false (nothing changed) if the pool is short.
  bool ensure(std::vector<int32_t>& table, int64_t length) {
    const int n = need(table, length);
    if (n > free_pages()) return false;
    for (int i = 0; i < n; ++i) {
      table.push_back(free_.top());
      free_.pop();
    }
    return true;
  }
  // Free pages holding no position below `length`.
  void truncate(std::vector<int32_t>& table, int64_t length) {
    const int keep = pages_for(length);
    while (static_cast<int>(table.size()) > keep) {
      free_.push(table.back());
      table.pop_back();
    }
  }
  int32_t slot(const std::vector<int32_t>& table, int64_t pos) const {
    return table[pos / page_size_] * page_size_ + static_cast<int32_t>(pos % page_size_);
  }

 private:
  int page_size_ = 16;
  int num_pages_ = 0;
  std::priority_queue<int32_t, std::vector<int32_t>, std::greater<int32_t>> free_;
};

}  // namespace spec
