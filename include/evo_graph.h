/*
 * evo_graph.h -- a shape-keyed cache of captured HIP graphs.
 *
 * ScaleFold (arXiv 2404.11068), Section 3.2, "CUDA Graph": once data
 * parallelism shrinks each GPU's work, the host-side cost of launching
 * thousands of small kernels per step shows; capturing the step into a graph
 * and replaying it removes that cost, and because recycling changes the
 * sequence of kernels between steps, the paper keeps a cache of graphs, one
 * per scenario.  This is that cache for HIP: the caller supplies a key (for
 * example a hash of the shapes and buffer addresses) and a function that
 * enqueues the step's work on a stream; on a miss the library captures the
 * function into a graph, instantiates it and keeps it; on every call it
 * launches the graph for the key.
 *
 * Rules for the record function: it runs once per key, while `stream` is
 * being captured (thread-local capture mode); it must only enqueue
 * asynchronous work on that stream (kernels of this library, copies between
 * device buffers) and must not allocate, free or synchronise.  Every replay
 * reads and writes the buffers the recorded work used, so callers keep their
 * inputs and outputs at fixed addresses (static buffers) per key.
 *
 * The cache owns host-side graph objects (and whatever the HIP runtime keeps
 * for them); it allocates no device memory of its own.  Not thread-safe: one
 * thread per cache.  Status codes are those of evo_attn.h (EVO_ERR_HIP when
 * capture, instantiation or launch fails; nothing is kept for the key then).
 */
#ifndef EVO_GRAPH_H
#define EVO_GRAPH_H

#include "evo_attn.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct evo_graph_cache evo_graph_cache;
typedef void (*evo_graph_record_fn)(void *user, void *stream);

/* capacity >= 1: at most that many graphs are kept; on overflow the least
 * recently used one is destroyed. */
int evo_graph_cache_create(int32_t capacity, evo_graph_cache **out);
int evo_graph_cache_destroy(evo_graph_cache *cache);

/* Launch the graph for `key` on `stream` (a hipStream_t, not NULL: the null
 * stream cannot be captured), capturing `record(user, stream)` first if the
 * key is new.  *captured (if not NULL) is set to 1 when this call captured. */
int evo_graph_cache_run(evo_graph_cache *cache, uint64_t key, evo_graph_record_fn record, void *user,
                        void *stream, int32_t *captured);

/* Number of graphs held; -1 for a NULL cache. */
int32_t evo_graph_cache_size(const evo_graph_cache *cache);

/* Destroy every graph (for example after the buffers they use were freed). */
int evo_graph_cache_clear(evo_graph_cache *cache);

#ifdef __cplusplus
}
#endif

#endif /* EVO_GRAPH_H */
