// evo_graph.cpp -- the shape-keyed HIP graph cache declared in
// include/evo_graph.h.
#include "evo_graph.h"

#include <hip/hip_runtime.h>

#include <list>
#include <unordered_map>

struct evo_graph_cache {
    struct Entry {
        uint64_t key;
        hipGraph_t graph;
        hipGraphExec_t exec;
    };
    int32_t capacity = 1;
    std::list<Entry> lru;  // most recently used first
    std::unordered_map<uint64_t, std::list<Entry>::iterator> index;

    static void release(Entry &e) {
        if (e.exec) (void)hipGraphExecDestroy(e.exec);
        if (e.graph) (void)hipGraphDestroy(e.graph);
        e.exec = nullptr;
        e.graph = nullptr;
    }
    void clear() {
        for (auto &e : lru) release(e);
        lru.clear();
        index.clear();
    }
};

extern "C" {

int evo_graph_cache_create(int32_t capacity, evo_graph_cache **out) {
    if (!out || capacity < 1) return EVO_ERR_INVALID_ARG;
    evo_graph_cache *c = new (std::nothrow) evo_graph_cache;
    if (!c) return EVO_ERR_HIP;
    c->capacity = capacity;
    *out = c;
    return EVO_OK;
}

int evo_graph_cache_destroy(evo_graph_cache *cache) {
    if (!cache) return EVO_ERR_INVALID_ARG;
    cache->clear();
    delete cache;
    return EVO_OK;
}

int32_t evo_graph_cache_size(const evo_graph_cache *cache) { return cache ? (int32_t)cache->lru.size() : -1; }

int evo_graph_cache_clear(evo_graph_cache *cache) {
    if (!cache) return EVO_ERR_INVALID_ARG;
    cache->clear();
    return EVO_OK;
}

int evo_graph_cache_run(evo_graph_cache *cache, uint64_t key, evo_graph_record_fn record, void *user, void *stream,
                        int32_t *captured) {
    if (!cache || !record || !stream) return EVO_ERR_INVALID_ARG;
    if (captured) *captured = 0;
    hipStream_t s = (hipStream_t)stream;
    auto it = cache->index.find(key);
    if (it == cache->index.end()) {
        evo_graph_cache::Entry e{key, nullptr, nullptr};
        (void)hipGetLastError();  // start from a clean error state
        if (hipStreamBeginCapture(s, hipStreamCaptureModeThreadLocal) != hipSuccess) return EVO_ERR_HIP;
        record(user, stream);
        const hipError_t rec_err = hipGetLastError();
        const hipError_t end_err = hipStreamEndCapture(s, &e.graph);
        if (rec_err != hipSuccess || end_err != hipSuccess || !e.graph) {
            evo_graph_cache::release(e);
            return EVO_ERR_HIP;
        }
        if (hipGraphInstantiate(&e.exec, e.graph, nullptr, nullptr, 0) != hipSuccess) {
            evo_graph_cache::release(e);
            return EVO_ERR_HIP;
        }
        if ((int32_t)cache->lru.size() >= cache->capacity) {
            evo_graph_cache::Entry &old = cache->lru.back();
            cache->index.erase(old.key);
            evo_graph_cache::release(old);
            cache->lru.pop_back();
        }
        cache->lru.push_front(e);
        it = cache->index.emplace(key, cache->lru.begin()).first;
        if (captured) *captured = 1;
    } else if (it->second != cache->lru.begin()) {
        cache->lru.splice(cache->lru.begin(), cache->lru, it->second);
    }
    return hipGraphLaunch(cache->lru.front().exec, s) == hipSuccess ? EVO_OK : EVO_ERR_HIP;
}

}  // extern "C"
