// Replacement model of the context cache (CPU): replays request traces through
// a size-limited cache under FIFO, LRU or Least Carbon Savings (GreenCache §5.5,
// Eq. 7 and Eq. 8). The cache model and the exact score arithmetic are stated in
// include/greencache_ctl.h.
#include "greencache_ctl.h"

#include <cmath>
#include <cstdint>
#include <new>
#include <set>
#include <unordered_map>
#include <utility>
#include <vector>

namespace {

struct Entry {
    int64_t tokens = 0;
    int64_t hits = 0;
    int64_t acc_tokens = 0;
    int32_t turn = 0;
    double t_insert = 0.0;
    double t_last = 0.0;
};

constexpr double kMinAge = 1e-6;

}  // namespace

struct gc_cache {
    int32_t policy;
    int64_t capacity;
    int64_t bytes_per_token;
    int64_t bytes = 0;
    double last_time = -INFINITY;
    std::unordered_map<int64_t, Entry> entries;
    // FIFO and LRU keep their order in a set of (time, key); LCS scores depend on
    // the current time, so they are recomputed over all entries at each eviction
    std::set<std::pair<double, int64_t>> order;
    gc_cache_stats stats{};

    int64_t size_of(const Entry& e) const { return e.tokens * bytes_per_token; }
    double order_time(const Entry& e) const { return policy == GC_POLICY_FIFO ? e.t_insert : e.t_last; }

    double score(const Entry& e, double now) const {
        const double age = std::fmax(now - e.t_insert, kMinAge);
        const double size = (double)size_of(e);
        if (policy == GC_POLICY_LCS) return ((double)e.acc_tokens * (double)e.hits) / (size * age);
        return ((double)e.turn * (double)e.acc_tokens) / (size * age);
    }

    // The entry to evict next at time `now` (never `keep` when has_keep); entries.end() if none.
    std::unordered_map<int64_t, Entry>::iterator victim(bool has_keep, int64_t keep, double now) {
        if (policy == GC_POLICY_FIFO || policy == GC_POLICY_LRU) {
            for (const auto& tk : order)
                if (!has_keep || tk.second != keep) return entries.find(tk.second);
            return entries.end();
        }
        auto best = entries.end();
        double bs = 0.0;
        for (auto itr = entries.begin(); itr != entries.end(); ++itr) {
            if (has_keep && itr->first == keep) continue;
            const double s = score(itr->second, now);
            if (best == entries.end() || s < bs ||
                (s == bs && (itr->second.t_insert < best->second.t_insert ||
                             (itr->second.t_insert == best->second.t_insert && itr->first < best->first)))) {
                best = itr;
                bs = s;
            }
        }
        return best;
    }

    void erase(std::unordered_map<int64_t, Entry>::iterator itr) {
        if (policy == GC_POLICY_FIFO || policy == GC_POLICY_LRU) order.erase({order_time(itr->second), itr->first});
        bytes -= size_of(itr->second);
        entries.erase(itr);
    }

    // Evict by the policy until the cached bytes fit. With has_keep, the entry `keep`
    // (the one just inserted or grown) is never chosen; if it alone exceeds the
    // capacity it is removed instead and nothing else is evicted for it.
    void fit(bool has_keep, int64_t keep, double now) {
        if (has_keep) {
            auto self = entries.find(keep);
            if (self != entries.end() && size_of(self->second) > capacity) {
                erase(self);
                ++stats.evictions;
            }
        }
        while (bytes > capacity) {
            auto v = victim(has_keep, keep, now);
            if (v == entries.end()) break;
            erase(v);
            ++stats.evictions;
        }
    }

    void touch_order(int64_t key, const Entry& before, const Entry& after) {
        if (policy == GC_POLICY_FIFO || policy == GC_POLICY_LRU) {
            order.erase({order_time(before), key});
            order.insert({order_time(after), key});
        }
    }

    int64_t access(const gc_request& q) {
        ++stats.requests;
        stats.prompt_tokens += q.prompt_tokens;
        const double now = q.time;
        last_time = now;
        auto itr = entries.find(q.key);
        int64_t reused = 0;
        if (itr != entries.end()) {
            Entry& e = itr->second;
            const Entry before = e;
            reused = q.context_tokens < e.tokens ? q.context_tokens : e.tokens;
            ++stats.hits;
            stats.reused_tokens += reused;
            e.hits += 1;
            e.acc_tokens += reused;
            e.turn = q.turn;
            e.t_last = now;
            if (q.total_tokens > e.tokens) {
                bytes += (q.total_tokens - e.tokens) * bytes_per_token;
                e.tokens = q.total_tokens;
            }
            touch_order(q.key, before, e);
        } else {
            Entry e;
            e.tokens = q.total_tokens;
            e.turn = q.turn;
            e.t_insert = now;
            e.t_last = now;
            entries.emplace(q.key, e);
            if (policy == GC_POLICY_FIFO || policy == GC_POLICY_LRU) order.insert({order_time(e), q.key});
            bytes += size_of(e);
            ++stats.insertions;
        }
        fit(true, q.key, now);
        return reused;
    }
};

extern "C" {

__attribute__((visibility("default")))
gc_ctl_status gc_cache_create(int32_t policy, int64_t capacity_bytes, int64_t bytes_per_token,
                              gc_cache** out) {
    if (out == nullptr) return GC_CTL_ERR_NULL_ARG;
    if (policy < GC_POLICY_FIFO || policy > GC_POLICY_LCS_MULTITURN || capacity_bytes < 0 ||
        bytes_per_token <= 0)
        return GC_CTL_ERR_BAD_ARG;
    gc_cache* c = new (std::nothrow) gc_cache();
    if (c == nullptr) return GC_CTL_ERR_NOMEM;
    c->policy = policy;
    c->capacity = capacity_bytes;
    c->bytes_per_token = bytes_per_token;
    *out = c;
    return GC_CTL_OK;
}

__attribute__((visibility("default")))
void gc_cache_destroy(gc_cache* cache) { delete cache; }

__attribute__((visibility("default")))
gc_ctl_status gc_cache_replay(gc_cache* cache, const gc_request* requests, int64_t n, int64_t* reused) {
    if (cache == nullptr) return GC_CTL_ERR_NULL_ARG;
    if (n < 0) return GC_CTL_ERR_BAD_ARG;
    if (n > 0 && requests == nullptr) return GC_CTL_ERR_NULL_ARG;
    double t = cache->last_time;
    for (int64_t i = 0; i < n; ++i) {
        const gc_request& q = requests[i];
        if (q.context_tokens < 0 || q.prompt_tokens < q.context_tokens || q.total_tokens < q.prompt_tokens ||
            q.turn < 0 || q.reserved != 0 || !std::isfinite(q.time) || q.time < t)
            return GC_CTL_ERR_BAD_ARG;
        t = q.time;
    }
    try {
        for (int64_t i = 0; i < n; ++i) {
            const int64_t r = cache->access(requests[i]);
            if (reused != nullptr) reused[i] = r;
        }
    } catch (const std::bad_alloc&) {
        return GC_CTL_ERR_NOMEM;
    }
    return GC_CTL_OK;
}

__attribute__((visibility("default")))
gc_ctl_status gc_cache_resize(gc_cache* cache, int64_t capacity_bytes, double now) {
    if (cache == nullptr) return GC_CTL_ERR_NULL_ARG;
    if (capacity_bytes < 0 || !std::isfinite(now) || now < cache->last_time) return GC_CTL_ERR_BAD_ARG;
    cache->capacity = capacity_bytes;
    cache->last_time = now;
    cache->fit(false, 0, now);
    return GC_CTL_OK;
}

__attribute__((visibility("default")))
gc_ctl_status gc_cache_get_stats(const gc_cache* cache, gc_cache_stats* stats) {
    if (cache == nullptr || stats == nullptr) return GC_CTL_ERR_NULL_ARG;
    *stats = cache->stats;
    stats->entries = (int64_t)cache->entries.size();
    stats->bytes = cache->bytes;
    return GC_CTL_OK;
}

__attribute__((visibility("default")))
gc_ctl_status gc_cache_keys(const gc_cache* cache, int64_t* keys, int64_t n, int64_t* count) {
    if (cache == nullptr || count == nullptr || (n > 0 && keys == nullptr)) return GC_CTL_ERR_NULL_ARG;
    std::vector<int64_t> all;
    all.reserve(cache->entries.size());
    for (const auto& kv : cache->entries) all.push_back(kv.first);
    std::set<int64_t> sorted(all.begin(), all.end());
    int64_t i = 0;
    for (int64_t k : sorted) {
        if (i >= n) break;
        keys[i++] = k;
    }
    *count = (int64_t)cache->entries.size();
    return GC_CTL_OK;
}

}  // extern "C"
