// Least-recently-used cache of per-work-list schedules, keyed by the work
// list's contents.  Host code only.
//
// Entries are reference counted: get() hands the caller its own reference,
// which the caller keeps until the kernels that read the entry are enqueued.
// An entry evicted by another thread in the meantime is destroyed (its
// device buffer freed) only when the last reference goes, so no launch ever
// reads a freed schedule.  Building an entry and every change of the map
// happen under one mutex.
#pragma once

#include <cstddef>
#include <list>
#include <memory>
#include <mutex>
#include <string>
#include <unordered_map>
#include <utility>

namespace nsp {

template <class Entry>
class LruCache {
 public:
  using Ptr = std::shared_ptr<const Entry>;

  explicit LruCache(size_t capacity) : cap_(capacity < 1 ? 1 : capacity) {}

  // The entry of `key` in *out.  On a miss, build(&ptr) creates it (returning
  // 0, or a nonzero status that get() returns without inserting anything).
  template <class Build>
  int get(const std::string &key, Ptr *out, Build build) {
    std::lock_guard<std::mutex> lock(mu_);
    auto it = map_.find(key);
    if (it != map_.end()) {
      lru_.splice(lru_.begin(), lru_, it->second.second);
      *out = it->second.first;
      return 0;
    }
    Ptr e;
    const int st = build(&e);
    if (st != 0) return st;
    while (map_.size() >= cap_) {
      map_.erase(lru_.back());   // the entry lives on while a caller still holds it
      lru_.pop_back();
    }
    lru_.push_front(key);
    map_.emplace(key, std::make_pair(e, lru_.begin()));
    *out = std::move(e);
    return 0;
  }

  size_t size() {
    std::lock_guard<std::mutex> lock(mu_);
    return map_.size();
  }

 private:
  std::mutex mu_;
  std::list<std::string> lru_;   // most recent at the front
  std::unordered_map<std::string, std::pair<Ptr, std::list<std::string>::iterator>> map_;
  size_t cap_;
};

}  // namespace nsp
