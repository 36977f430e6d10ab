// Bounded least-recently-used cache of the device-resident work plans, with
// stream-safe retirement of evicted entries. Host code only (no HIP calls: the
// device side is a policy), so the bookkeeping is testable without a GPU.
//
// A cached value is in use while a caller holds it between acquire() and
// release() (the host part of a call: from the cache lookup to the enqueue of its
// kernels) and while kernels enqueued with it may still run, which the policy
// tracks (Ops::idle, e.g. events recorded after the launches). Evicting a value
// only moves it to a retired list; collect() frees retired values once no caller
// holds them and Ops::idle says their work is done. A pinned value (one captured
// into a graph, which may replay at any later time) is never evicted.
#pragma once

#include <cstddef>
#include <list>
#include <string>
#include <unordered_map>
#include <utility>

namespace ta {

// Ops must provide:
//   bool idle(Value&)     no enqueued work may still read the value
//   void release(Value&)  free the value's resources (called exactly once)
template <class Value, class Ops>
class PlanCache {
 public:
  struct Slot {
    std::string key;
    Value value;
    int holders = 0;      // callers between acquire() and release()
    bool pinned = false;  // never evicted
  };
  using Handle = Slot*;

  explicit PlanCache(size_t capacity, Ops ops = Ops()) : cap_(capacity ? capacity : 1), ops_(ops) {}
  PlanCache(const PlanCache&) = delete;
  PlanCache& operator=(const PlanCache&) = delete;
  ~PlanCache() = default;  // process-lifetime object: device memory is left to the driver

  // The live slot for key, marked most recently used and held by the caller, or null.
  Handle acquire(const std::string& key) {
    auto it = index_.find(key);
    if (it == index_.end()) return nullptr;
    live_.splice(live_.begin(), live_, it->second);
    ++it->second->holders;
    return &*it->second;
  }

  // Inserts a new value for key (not present), held by the caller. Entries beyond the
  // capacity are evicted least recently used first, skipping held and pinned ones.
  Handle insert(std::string key, Value value) {
    live_.push_front(Slot{std::move(key), std::move(value), 1, false});
    index_[live_.front().key] = live_.begin();
    evict_beyond_capacity();
    collect();
    return &live_.front();
  }

  // The caller is done enqueuing work with h (its completion is the policy's business).
  void release(Handle h) {
    if (h && h->holders > 0) --h->holders;
  }

  void pin(Handle h) {
    if (h) h->pinned = true;
  }

  // Frees retired values that nobody holds and whose work is done.
  void collect() {
    for (auto it = retired_.begin(); it != retired_.end();) {
      if (it->holders == 0 && ops_.idle(it->value)) {
        ops_.release(it->value);
        it = retired_.erase(it);
      } else {
        ++it;
      }
    }
  }

  size_t size() const { return live_.size(); }
  size_t retired() const { return retired_.size(); }
  size_t capacity() const { return cap_; }
  Ops& ops() { return ops_; }

 private:
  void evict_beyond_capacity() {
    auto it = live_.end();
    while (live_.size() > cap_ && it != live_.begin()) {
      --it;
      if (it->holders > 0 || it->pinned) continue;
      index_.erase(it->key);
      auto victim = it++;  // keep the scan position valid across the splice
      retired_.splice(retired_.end(), live_, victim);
    }
  }

  size_t cap_;
  Ops ops_;
  std::list<Slot> live_;  // most recently used first
  std::list<Slot> retired_;
  std::unordered_map<std::string, typename std::list<Slot>::iterator> index_;
};

}  // namespace ta
