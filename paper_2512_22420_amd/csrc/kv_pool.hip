// Contraction of the elastic KV pool (Sec. 6.4): the migration plan over the
// block tables (host) and the block migration kernel (device).
#include <string.h>

#include <unordered_map>
#include <unordered_set>
#include <vector>

#include "../../include/nightjar.h"
#include "../../include/nightjar_memory.h"
#include "common.h"
#include "kernels.h"

namespace nj {
namespace {

constexpr int kMigrateLayers = 64;  // layers per launch (page pointers travel in the kernel arguments)
constexpr int kMigrateThreads = 256;
constexpr int kMigrateUnroll = 8;   // 16-byte loads in flight per thread before its stores

struct LayerPages {
  u32x4* k[kMigrateLayers];
  u32x4* v[kMigrateLayers];
};

// grid (moves, layers of this launch): workgroup (i, l) copies block src[i] ->
// dst[i] of layer l0 + l, K then V, as `units` 16-byte pieces each (one block
// of one layer is contiguous in both page layouts).  Every thread issues
// kMigrateUnroll loads before its stores.
__global__ __launch_bounds__(kMigrateThreads) void kv_migrate_kernel(LayerPages pages, const int32_t* __restrict__ src,
                                                                     const int32_t* __restrict__ dst, int units,
                                                                     int num_blocks, int* __restrict__ err) {
  const int i = blockIdx.x, l = blockIdx.y;
  const int s = src[i], d = dst[i];
  if (s < 0 || s >= num_blocks || d < 0 || d >= num_blocks) {
    if (threadIdx.x == 0 && l == 0 && err) flag_error(err, kErrBlock);
    return;
  }
  const u32x4* ks = pages.k[l] + (size_t)s * units;
  const u32x4* vs = pages.v[l] + (size_t)s * units;
  u32x4* kd = pages.k[l] + (size_t)d * units;
  u32x4* vd = pages.v[l] + (size_t)d * units;
  const int total = 2 * units;  // K pieces, then V pieces
  for (int base = 0; base < total; base += kMigrateThreads * kMigrateUnroll) {
    u32x4 buf[kMigrateUnroll];
#pragma unroll
    for (int r = 0; r < kMigrateUnroll; ++r) {
      const int u = base + r * kMigrateThreads + threadIdx.x;
      if (u < total) buf[r] = u < units ? ks[u] : vs[u - units];
    }
#pragma unroll
    for (int r = 0; r < kMigrateUnroll; ++r) {
      const int u = base + r * kMigrateThreads + threadIdx.x;
      if (u < total) {
        if (u < units) kd[u] = buf[r];
        else vd[u - units] = buf[r];
      }
    }
  }
}

}  // namespace
}  // namespace nj

using namespace nj;

extern "C" {

int nightjar_contraction_plan(int32_t* block_table, int32_t B, int32_t max_blocks, const int32_t* free_list,
                              int32_t n_free, int32_t k_boundary, int32_t k_total, int32_t* src, int32_t* dst,
                              int32_t cap, int32_t* n_moves, int32_t* new_free, int32_t* n_new_free) {
  if (!block_table || !src || !dst || !n_moves || !new_free || !n_new_free || (n_free > 0 && !free_list))
    return set_last_error(NJ_EINVAL, "contraction_plan: NULL pointer");
  if (B < 0 || max_blocks < 0 || n_free < 0 || cap < 0 || k_boundary < 0 || k_boundary > k_total)
    return set_last_error(NJ_EINVAL, "contraction_plan: bad sizes (need 0 <= k_boundary <= k_total)");
  const size_t entries = (size_t)B * max_blocks;
  // Step 1: live blocks in the reclaimed region, in order of first appearance
  std::vector<int32_t> evict;
  std::unordered_map<int32_t, int32_t> slot;  // old id -> index in evict
  std::unordered_set<int32_t> live;
  for (size_t e = 0; e < entries; ++e) {
    const int32_t id = block_table[e];
    if (id < 0) continue;
    if (id >= k_total) return set_last_error(NJ_EINVAL, "contraction_plan: table entry %d >= k_total %d", id, k_total);
    live.insert(id);
    if (id >= k_boundary && !slot.count(id)) {
      slot.emplace(id, (int32_t)evict.size());
      evict.push_back(id);
    }
  }
  std::unordered_set<int32_t> seen;
  for (int i = 0; i < n_free; ++i) {
    const int32_t id = free_list[i];
    if (id < 0 || id >= k_total) return set_last_error(NJ_EINVAL, "contraction_plan: free id %d outside [0, k_total)", id);
    if (!seen.insert(id).second) return set_last_error(NJ_EINVAL, "contraction_plan: free id %d listed twice", id);
    if (live.count(id)) return set_last_error(NJ_EINVAL, "contraction_plan: free id %d is used by a table", id);
  }
  if ((int64_t)evict.size() > cap)
    return set_last_error(NJ_EINVAL, "contraction_plan: %zu moves exceed cap %d", evict.size(), cap);
  // Step 2: destinations from the free list below the boundary, in its order
  std::vector<int32_t> dsts;
  std::vector<char> taken(n_free, 0);
  for (int i = 0; i < n_free && dsts.size() < evict.size(); ++i)
    if (free_list[i] < k_boundary) {
      dsts.push_back(free_list[i]);
      taken[i] = 1;
    }
  if (dsts.size() < evict.size())
    return set_last_error(NJ_EAGAIN, "contraction_plan: %zu live blocks above the boundary, %zu free blocks below it",
                          evict.size(), dsts.size());
  for (size_t m = 0; m < evict.size(); ++m) {
    src[m] = evict[m];
    dst[m] = dsts[m];
  }
  *n_moves = (int32_t)evict.size();
  // Step 3: remap the tables
  for (size_t e = 0; e < entries; ++e) {
    const int32_t id = block_table[e];
    if (id >= k_boundary) block_table[e] = dsts[slot[id]];
  }
  // Step 5: the free list without the destinations and the reclaimed region
  int32_t nf = 0;
  for (int i = 0; i < n_free; ++i)
    if (!taken[i] && free_list[i] < k_boundary) new_free[nf++] = free_list[i];
  *n_new_free = nf;
  return NJ_OK;
}

int nightjar_kv_migrate(const nj_model_desc* desc, const nj_kv_cache* kv, const int32_t* src, const int32_t* dst,
                        int32_t n, int32_t* device_error, void* stream) {
  if (!desc || !kv || !kv->k_pages || !kv->v_pages) return set_last_error(NJ_EINVAL, "kv_migrate: NULL desc or cache");
  const nj_model_desc& d = *desc;
  if (d.n_layers < 1 || d.n_kv_heads < 1 || d.head_dim < 8 || d.head_dim % 8 || d.block_size != 16 ||
      (d.dtype != NJ_F32 && d.dtype != NJ_BF16) || kv->num_blocks < 1)
    return set_last_error(NJ_EINVAL, "kv_migrate: bad descriptor or num_blocks");
  if (n < 0 || (n > 0 && (!src || !dst))) return set_last_error(NJ_EINVAL, "kv_migrate: bad n or NULL map");
  if (n > (1 << 24)) return set_last_error(NJ_EINVAL, "kv_migrate: more than 2^24 moves in one call");
  for (int l = 0; l < d.n_layers; ++l)
    if (!kv->k_pages[l] || !kv->v_pages[l] || ((uintptr_t)kv->k_pages[l] & 15) || ((uintptr_t)kv->v_pages[l] & 15))
      return set_last_error(NJ_EINVAL, "kv_migrate: layer %d pages NULL or not 16-byte aligned", l);
  hipStream_t s = (hipStream_t)stream;
  hipError_t e = hipSuccess;
  if (device_error) e = launch_fill_i32(device_error, 0, 1, s);
  if (e != hipSuccess) return set_last_error(NJ_EHIP, "kv_migrate: %s", hipGetErrorString(e));
  if (n == 0) return NJ_OK;
  const size_t elt = d.dtype == NJ_BF16 ? 2 : 4;
  const int units = (int)((size_t)d.n_kv_heads * 16 * d.head_dim * elt / 16);
  for (int l0 = 0; l0 < d.n_layers; l0 += kMigrateLayers) {
    const int nl = std::min(kMigrateLayers, d.n_layers - l0);
    LayerPages p{};
    for (int i = 0; i < nl; ++i) {
      p.k[i] = static_cast<u32x4*>(kv->k_pages[l0 + i]);
      p.v[i] = static_cast<u32x4*>(kv->v_pages[l0 + i]);
    }
    hipLaunchKernelGGL(kv_migrate_kernel, dim3(n, nl), dim3(kMigrateThreads), 0, s, p, src, dst, units,
                       kv->num_blocks, device_error);
    e = hipGetLastError();
    if (e != hipSuccess) return set_last_error(NJ_EHIP, "kv_migrate: %s", hipGetErrorString(e));
  }
  return NJ_OK;
}

}  // extern "C"
