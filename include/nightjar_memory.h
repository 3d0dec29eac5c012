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

#ifdef __cplusplus
}
#endif

#endif /* NIGHTJAR_MEMORY_H */
