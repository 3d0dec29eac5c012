/*
 * nightjar_memory.h -- elastic KV-cache pool of Nightjar (arXiv 2512.22420,
 * Sec. 6): contraction of an expanded pool (Sec. 6.4, Steps 1-5) and the
 * vectorised block migration it needs, on MI355X.  Part of libnightjar.so;
 * conventions (return codes, nightjar_last_error, streams, page layouts) as in
 * nightjar.h.
 *
 * When the draft model is offloaded the KV pool grows past its baseline
 * capacity: physical blocks [K_boundary, K_total) are added (Sec. 6.3).  To
 * give that memory back (before the draft model is reloaded) every live block
 * with an id >= K_boundary is moved to a free block below the boundary and the
 * block tables are rewritten; the attention reads blocks only through the
 * tables, so decoding is unaffected (Sec. 6.4, Sec. 6.5).
 */
#ifndef NIGHTJAR_MEMORY_H
#define NIGHTJAR_MEMORY_H

#include <stddef.h>
#include <stdint.h>

#include "nightjar.h"

#ifdef __cplusplus
extern "C" {
#endif

enum {
  NJ_EAGAIN = -4 /* not possible now (e.g. too few free blocks below the boundary); nothing was changed */
};

/*
 * nightjar_contraction_plan -- Steps 1, 2, 3 and 5 of the contraction, on host
 * memory (the allocator's state lives on the host).
 *
 *   block_table   host int32 [B][max_blocks], in/out: entry j of row b is a
 *                 physical block id, or < 0 for an unused entry; every entry
 *                 >= k_boundary is rewritten to its new id (Step 3)
 *   free_list     host int32 [n_free]: the allocator's free physical blocks,
 *                 in allocation order
 *   k_boundary    first id of the region being reclaimed
 *   src, dst      host int32 [cap], out: the migration map M (Step 2), one
 *                 pair per distinct live block >= k_boundary, in order of first
 *                 appearance in the tables (row-major); a block shared by
 *                 several rows moves once.  dst ids are taken from free_list in
 *                 its order, skipping ids >= k_boundary.
 *   n_moves       out: number of pairs
 *   new_free      host int32 [n_free], out: the free list after contraction
 *                 (Step 5): free_list in its order minus the blocks taken as
 *                 destinations and minus every id >= k_boundary
 *   n_new_free    out
 * Returns NJ_OK; NJ_EAGAIN (nothing changed) when there are fewer free blocks
 * below the boundary than blocks to move (the caller defers the contraction,
 * Sec. 6.1 "drain-aware"); NJ_EINVAL for bad arguments (NULL, sizes, cap
 * smaller than the moves, an id >= k_total, duplicate free ids, a free block
 * that a table still uses).
 */
int nightjar_contraction_plan(int32_t* block_table, int32_t B, int32_t max_blocks, const int32_t* free_list,
                              int32_t n_free, int32_t k_boundary, int32_t k_total, int32_t* src, int32_t* dst,
                              int32_t cap, int32_t* n_moves, int32_t* new_free, int32_t* n_new_free);

/*
 * nightjar_kv_migrate -- Step 4: copy physical block src[i] to dst[i] in the K
 * and V pages of every layer (the whole block, all KV heads), asynchronously
 * on `stream`.  One workgroup per (move, layer) streams the block's K and V
 * (2 * Hkv * 16 * D elements) with 16-byte loads and stores.
 *
 *   desc, kv     the model descriptor (n_layers, n_kv_heads, head_dim, dtype)
 *                and the pages (16-byte aligned)
 *   src, dst     device int32 [n]: the migration map; dst ids distinct and no
 *                dst id among the src ids (as nightjar_contraction_plan makes them)
 *   device_error device int32, out (nullable): NJ_DEV_BAD_BLOCK if a pair had an
 *                id outside [0, num_blocks) (that pair is skipped); 0 otherwise
 * n == 0 enqueues nothing but the error word's clear.
 */
int nightjar_kv_migrate(const nj_model_desc* desc, const nj_kv_cache* kv, const int32_t* src, const int32_t* dst,
                        int32_t n, int32_t* device_error, void* stream);

/* ---------------------------------------------------------------------------
 * Elastic pool control (Sec. 6.1 trigger conditions, Sec. 6.2 asynchronous
 * offload and reload, Sec. 6.3 expansion, Sec. 6.4 contraction).  A host
 * state machine the serving loop calls once per scheduling step; it says when
 * to offload the draft model, grow the pool, shrink it back and reload the
 * draft, and how far the planner may speculate meanwhile.
 *
 * States: RESIDENT (draft weights on the GPU, pool of n_orig blocks),
 * OFFLOADING (draft copy to host in flight), OFFLOADED (draft on the host, pool
 * n_orig), EXPANDED (draft on the host, pool n_orig + n_draft: blocks
 * [n_orig, n_orig + n_draft) usable), CONTRACTING (live blocks of the extra
 * region being migrated below it), RELOADING (draft copy back in flight).
 * Speculation is allowed (gamma_allowed = 1) only in RESIDENT.
 *
 * Transitions (readings of Sec. 6.1, with its persistence windows):
 *   RESIDENT -> OFFLOADING (action OFFLOAD_DRAFT): speculation disabled
 *     (this step's gamma = 0) and n_free < tau_low, both for t_persist
 *     consecutive steps;
 *   OFFLOADING -> OFFLOADED: nightjar_elastic_done(OFFLOAD_DRAFT);
 *   OFFLOADED -> EXPANDED (action EXPAND, immediate): n_free < tau_low for
 *     t_persist consecutive steps (the steps before the offload count);
 *   EXPANDED -> CONTRACTING (action CONTRACT): no waiting requests and
 *     n_free > n_draft + tau_low, for reload_persist consecutive steps, and at
 *     most max_migrate live blocks above the boundary (drain-aware; otherwise
 *     deferred, the hysteresis keeps speculation off under load);
 *   CONTRACTING -> OFFLOADED: nightjar_elastic_done(CONTRACT), and the draft
 *     is reloaded at the next step (action RELOAD_DRAFT);
 *   OFFLOADED -> RELOADING (action RELOAD_DRAFT): the same low-load condition
 *     for reload_persist steps (or right after a contraction);
 *   RELOADING -> RESIDENT: nightjar_elastic_done(RELOAD_DRAFT).
 * n_free counts the free blocks of the current pool (n_orig, or
 * n_orig + n_draft when expanded).
 * ------------------------------------------------------------------------- */
enum {
  NJ_POOL_RESIDENT = 0,
  NJ_POOL_OFFLOADING = 1,
  NJ_POOL_OFFLOADED = 2,
  NJ_POOL_EXPANDED = 3,
  NJ_POOL_CONTRACTING = 4,
  NJ_POOL_RELOADING = 5
};
enum { NJ_ACT_NONE = 0, NJ_ACT_OFFLOAD_DRAFT = 1, NJ_ACT_EXPAND = 2, NJ_ACT_CONTRACT = 3, NJ_ACT_RELOAD_DRAFT = 4 };

typedef struct nj_elastic nj_elastic;
typedef struct nj_elastic_config {
  int32_t n_orig;         /* baseline KV blocks                                        */
  int32_t n_draft;        /* blocks the draft weights are worth: ceil(S_draft / B_block) */
  int32_t tau_low;        /* scarcity threshold, in free blocks                         */
  int32_t t_persist;      /* steps the low-memory state must last (the paper uses 3)    */
  int32_t reload_persist; /* steps the low-load state must last before shrinking/reload */
  int32_t max_migrate;    /* live blocks above the boundary a contraction may move      */
} nj_elastic_config;

nj_elastic* nightjar_elastic_create(const nj_elastic_config* cfg); /* NULL on a bad config */
void nightjar_elastic_destroy(nj_elastic* e);
/*
 * One scheduling step: the current pool's free blocks, the waiting-queue
 * length, whether this step speculates (gamma > 0), and the live blocks at or
 * above n_orig.  *action receives the action to start now (NJ_ACT_*).
 */
int nightjar_elastic_step(nj_elastic* e, int32_t n_free, int32_t n_waiting, int32_t speculating,
                          int32_t live_above, int32_t* action);
/* The asynchronous part of `action` has finished (OFFLOAD_DRAFT, CONTRACT or RELOAD_DRAFT). */
int nightjar_elastic_done(nj_elastic* e, int32_t action);
int nightjar_elastic_state(const nj_elastic* e, int32_t* state, int32_t* pool_blocks, int32_t* gamma_allowed);

/*
 * Draft weight offload and reload (Sec. 6.2): an asynchronous DMA copy of
 * `bytes` between device memory and pinned host memory (allocated with
 * hipHostMalloc, e.g. torch's pin_memory), on `stream` -- a side stream, so the
 * copy overlaps the decoding steps on the main one.  NJ_EINVAL for NULL
 * pointers; NJ_EHIP if the runtime refuses the copy.
 */
int nightjar_offload(const void* device_src, void* host_dst, size_t bytes, void* stream);
int nightjar_reload(const void* host_src, void* device_dst, size_t bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* NIGHTJAR_MEMORY_H */
