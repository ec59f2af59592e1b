// The KV store H of Appendix C: prefix key -> cache entry, FIFO eviction.
// Host-only and HIP-free, so it also builds with a plain C++ compiler.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <deque>
#include <unordered_map>

namespace bc {

struct CacheEntry {
  int m = 0;           // prefix tokens
  int n_layers = 0;    // Lc: layers whose prefix K/V are cached
  void* mem = nullptr; // caller-owned device memory of the entry
  size_t bytes = 0;
};

class CacheTable {
 public:
  explicit CacheTable(int capacity) : capacity_(capacity) {}

  int capacity() const { return capacity_; }
  size_t size() const { return map_.size(); }

  // O(1) hit test (hash map), as in the paper's lookup of h(p).
  const CacheEntry* find(uint64_t key) const {
    auto it = map_.find(key);
    return it == map_.end() ? nullptr : &it->second;
  }
  bool contains(uint64_t key) const { return map_.count(key) != 0; }

  // Inserts a key that is not present.  When the table was full the oldest
  // entry is evicted; returns true and sets *evicted_key in that case.  Every
  // allocation happens before anything is removed, so a failed one
  // (std::bad_alloc) leaves the table exactly as it was.
  bool insert(uint64_t key, const CacheEntry& e, uint64_t* evicted_key) {
    auto it = map_.emplace(key, e).first;
    try {
      order_.push_back(key);
    } catch (...) {
      map_.erase(it);
      throw;
    }
    if ((int)map_.size() <= capacity_) return false;
    const uint64_t old = order_.front();
    order_.pop_front();
    map_.erase(old);
    *evicted_key = old;
    return true;
  }

  bool erase(uint64_t key) {
    if (map_.erase(key) == 0) return false;
    for (auto it = order_.begin(); it != order_.end(); ++it)
      if (*it == key) {
        order_.erase(it);
        break;
      }
    return true;
  }

  // Keys oldest first (the eviction order).
  const std::deque<uint64_t>& order() const { return order_; }

 private:
  int capacity_;
  std::unordered_map<uint64_t, CacheEntry> map_;
  std::deque<uint64_t> order_;
};

// XXH64 of `len` bytes with `seed` (published xxHash64 algorithm).
uint64_t xxh64(const void* data, size_t len, uint64_t seed);

}  // namespace bc
