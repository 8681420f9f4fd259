/*
 * greencache_ctl.h - C ABI of the context cache's replacement model (CPU).
 *
 * GreenCache (arXiv 2505.23970) keeps the KV of earlier requests' context in
 * a size-limited cache and evicts, when space is needed or the cache shrinks,
 * the entries with the lowest score (§5.5 "Cache Manager and Replacement
 * Policy"). This library replays a request trace through such a cache under
 * one of the policies the paper compares (§6.3.2, "Replacement Policy
 * Comparison", Table tab:replacement): FIFO, LRU and Least Carbon Savings (LCS, Eq. 7, with the
 * multi-turn form of Eq. 8; the document form of Eq. 9 coincides with Eq. 7
 * here, see gc_policy). It holds no GPU code.
 *
 * Cache model (a reading of §5.5: the paper describes the policy, not the
 * bookkeeping):
 *   - One entry per key (a conversation or a document), holding the KV of
 *     `tokens` tokens; its size is tokens * bytes_per_token.
 *   - A request (key, turn, context_tokens, prompt_tokens, total_tokens, time)
 *     hits when its key is cached: it reuses min(context_tokens, tokens)
 *     tokens. The entry's hits grow by one, its accumulated reused tokens by
 *     that amount, its turn becomes the request's, its last access the
 *     request's time. Then the entry takes total_tokens tokens if that is
 *     more (the processed request's KV is saved, §2.2).
 *   - A miss reuses nothing and inserts the entry with total_tokens tokens,
 *     hits 0, accumulated tokens 0, inserted and last accessed at `time`.
 *   - Whenever the cached bytes exceed the capacity, other entries are
 *     evicted, lowest score first, until they fit; an entry that alone
 *     exceeds the capacity is removed instead (counted as an eviction) and
 *     nothing else is evicted for it.
 *   - Scores at time `now` (ties: earlier insertion first, then smaller key):
 *       FIFO: insertion time;  LRU: last access time;
 *       LCS (Eq. 7):           acc_tokens * hits / (size * age)
 *       LCS multi-turn (Eq. 8): turn * acc_tokens / (size * age)
 *     with size in bytes and age = max(now - insertion time, 1e-6) seconds;
 *     products and quotients in IEEE double in exactly this order.
 *   - Requests must come in non-decreasing time order.
 * Token hit rate (the paper's "cache hit rate", §6.3.2) = reused tokens / sum
 * of prompt_tokens.
 *
 * Conventions: all pointers belong to the caller; a gc_cache is not
 * thread-safe (one thread at a time). Errors leave the cache unchanged.
 */
#ifndef GREENCACHE_CTL_H
#define GREENCACHE_CTL_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum gc_ctl_status {
    GC_CTL_OK = 0,
    GC_CTL_ERR_NULL_ARG = -1,  /* a required pointer is NULL */
    GC_CTL_ERR_BAD_ARG = -2,   /* unknown policy, negative size or length, prompt < context,
                                  total < prompt, time going backwards, non-finite time */
    GC_CTL_ERR_NOMEM = -3      /* allocation failed */
} gc_ctl_status;

typedef enum gc_policy {
    GC_POLICY_FIFO = 0,
    GC_POLICY_LRU = 1,
    GC_POLICY_LCS = 2,            /* Eq. 7 (and Eq. 9: hits x reused document length) */
    GC_POLICY_LCS_MULTITURN = 3   /* Eq. 8 */
} gc_policy;

typedef struct gc_request {
    int64_t key;             /* conversation or document id */
    int64_t context_tokens;  /* leading tokens of the prompt that a cached entry can supply */
    int64_t prompt_tokens;   /* input tokens of the request (>= context_tokens) */
    int64_t total_tokens;    /* tokens the entry holds after the request (>= prompt_tokens) */
    int32_t turn;            /* turn (or question) number within the key, from 1 */
    int32_t reserved;        /* must be 0 */
    double time;             /* arrival time in seconds, non-decreasing */
} gc_request;

typedef struct gc_cache_stats {
    int64_t requests, hits, reused_tokens, prompt_tokens;
    int64_t insertions, evictions, entries, bytes;
} gc_cache_stats;

typedef struct gc_cache gc_cache;

/* A cache of capacity_bytes (>= 0) holding bytes_per_token (> 0) bytes per token. */
gc_ctl_status gc_cache_create(int32_t policy, int64_t capacity_bytes, int64_t bytes_per_token,
                              gc_cache** out);
void gc_cache_destroy(gc_cache* cache);

/* Replay n requests in order. reused[i] (if reused != NULL) receives the tokens
 * request i reused. The requests are validated before any of them is applied. */
gc_ctl_status gc_cache_replay(gc_cache* cache, const gc_request* requests, int64_t n,
                              int64_t* reused);

/* Set a new capacity at time `now` (the cache manager's resize, §5.5): when it
 * shrinks below the cached bytes, entries are evicted by the policy. */
gc_ctl_status gc_cache_resize(gc_cache* cache, int64_t capacity_bytes, double now);

/* Counters since creation (entries and bytes: current). */
gc_ctl_status gc_cache_get_stats(const gc_cache* cache, gc_cache_stats* stats);

/* Keys of the cached entries in ascending key order; writes min(n, entries)
 * keys and returns the number of entries in *count. */
gc_ctl_status gc_cache_keys(const gc_cache* cache, int64_t* keys, int64_t n, int64_t* count);

#ifdef __cplusplus
}
#endif

#endif /* GREENCACHE_CTL_H */
