// The work list of the bf16 paged attention: which (sequence, KV head, KV
// split) each workgroup of the attention grid takes.  Built once per step by
// one workgroup (the QKV GEMM's bookkeeping workgroup, or attn_plan_kernel)
// from the device context lengths; the attention reads one item per
// workgroup.
//
// Sequence b has nb_b = ceil(ctx_b / 16) cached blocks (ctx_b clamped as the
// attention clamps it).  With a split length of S blocks it gets
// s_b = max(1, ceil(nb_b / S)) splits per KV head, and items are numbered
// (b, KV head, split) in that order, so the splits of one (sequence, KV head)
// are consecutive and their partials sit in consecutive slots.  S is the
// smallest of kCand lengths spread over [s_lo, s_hi] whose item count fits the
// grid: s_lo = max(kMinSplitBlocks, ceil(Hkv * sum nb / nwg)) (no fewer
// items can fit), s_hi = max(s_lo, ceil(Hkv * sum nb / (nwg - pairs))), which
// always fits since sum_b ceil(nb_b / S) <= sum nb / S + B.  Items past the
// list are written with nsplit = 0 (that workgroup exits).
//
// The partials of a (sequence, KV head)'s splits sit in consecutive slots
// numbered in (b, KV head, split) order (slot0 of the item: its pair's first),
// but the items run in the order of the list, which, when the grid is more
// than one round of resident workgroups, puts the longest splits first
// (longest-processing-time order: short items left for last fill the final
// round instead of a long one holding it open).  Items of equal length take the
// order their sequences' atomic increments give them; which workgroup runs an
// item does not change its result.
#pragma once

#include <climits>

#include "common.h"

namespace nj {

#ifndef NJ_ATTN_MIN_SPLIT
#define NJ_ATTN_MIN_SPLIT 16
#endif
#ifndef NJ_ATTN_EXTRA_WGS
#define NJ_ATTN_EXTRA_WGS 512
#endif
constexpr int kMinSplitBlocks = NJ_ATTN_MIN_SPLIT;  // cached blocks a split holds at least
constexpr int kExtraWorkgroups = NJ_ATTN_EXTRA_WGS; // workgroups beyond one per (sequence, KV head), at most
constexpr int kExtraWorkgroupsLarge = 128;          // ... once the pairs fill half of the resident workgroups

struct AttnWork {
  int b, kvh, split, nsplit;  // nsplit == 0: no item for this workgroup
  int c0, c1;                 // the split's cached blocks [c0, c1)
  int ctx;                    // the sequence's context length clamped into the table, or its bitwise
                              // complement when the caller's length was out of range (flagged by split 0)
  int slot0;                  // partial slot of the pair's split 0
};
static_assert(sizeof(AttnWork) == 32, "one item is two 16-byte loads");
constexpr int kOrderBuckets = 256;  // split lengths (in blocks) the list orders by; longer ones share the last

__device__ __forceinline__ int attn_clamp_ctx(int c, int max_blocks, int T) {
  const int cap = max_blocks * kBlock - T;
  return (c < 0 || c > cap) ? max(0, min(c, cap)) : c;
}

// Run by all NT threads of one workgroup (every thread must call it).
// scratch: at least attn_work_scratch_ints(NT) ints of LDS, not otherwise in use.
__host__ __device__ constexpr int attn_work_scratch_ints(int NT) { return 8 * (NT / 64) + 3 * NT / 2 + kOrderBuckets; }
template <int NT>
__device__ void build_attn_work(const int32_t* __restrict__ ctx, int B, int Hkv, int T, int max_blocks, int nwg,
                                bool order, AttnWork* __restrict__ work, int* scratch) {
  constexpr int kCand = 8, NWV = NT / 64;
  constexpr int kKeep = 4;  // context lengths a thread keeps in registers (more are re-read)
  const int per = (B + NT - 1) / NT;
  const int b0 = min(B, (int)threadIdx.x * per), b1 = min(B, b0 + per);
  const int lane = threadIdx.x & 63, wave = threadIdx.x / 64;
  int* s_red = scratch;                // [NWV][kCand]
  int* s_seq = scratch + NWV * kCand;  // small batches: [B][3] first slot, context, first list position
  int* s_hist = s_seq + 3 * NT / 2;    // [kOrderBuckets] items per split-length bucket, then list cursors
  auto nblocks_raw = [&](int raw) { return (attn_clamp_ctx(raw, max_blocks, T) + kBlock - 1) / kBlock; };
  auto wsum = [](int v) {
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
    return v;
  };
  auto bucket = [&](int n, int sb) {    // longest splits first
    return kOrderBuckets - 1 - min((n + sb - 1) / sb, kOrderBuckets - 1);
  };
  // Exclusive scan of s_hist into list positions (every thread calls it).
  auto scan_hist = [&]() {
    __syncthreads();
    if (wave == 0) {
      constexpr int PER = kOrderBuckets / 64;
      int h[PER], sum = 0;
#pragma unroll
      for (int e = 0; e < PER; ++e) sum += (h[e] = s_hist[lane * PER + e]);
      int incl = sum;
      for (int o = 1; o < 64; o <<= 1) {
        const int up = __shfl_up(incl, o);
        if (lane >= o) incl += up;
      }
      int run = incl - sum;
#pragma unroll
      for (int e = 0; e < PER; ++e) {
        s_hist[lane * PER + e] = run;
        run += h[e];
      }
    }
    __syncthreads();
  };
  // Small batches (B <= NT / 2, s_seq holding each sequence's first slot and
  // context): list positions, then the items, NT / B threads per sequence.
  auto put_small = [&](int S) {
    if (order) {
      for (int i = threadIdx.x; i < kOrderBuckets; i += NT) s_hist[i] = 0;
      __syncthreads();
      int n = 0, sb = 0;
      if ((int)threadIdx.x < B) {
        n = nblocks_raw(s_seq[3 * threadIdx.x + 1]);
        sb = max(1, (n + S - 1) / S);
        atomicAdd(&s_hist[bucket(n, sb)], Hkv * sb);
      }
      scan_hist();
      if ((int)threadIdx.x < B) s_seq[3 * threadIdx.x + 2] = atomicAdd(&s_hist[bucket(n, sb)], Hkv * sb);
      __syncthreads();
    }
    const int tps = NT / B, b = threadIdx.x / tps, j = threadIdx.x % tps;
    if (b < B) {
      const int slot = s_seq[3 * b], raw = s_seq[3 * b + 1], pos = order ? s_seq[3 * b + 2] : slot;
      const int c = attn_clamp_ctx(raw, max_blocks, T), nb = (c + kBlock - 1) / kBlock;
      const int sbb = max(1, (nb + S - 1) / S);
      for (int q = j; q < Hkv * sbb; q += tps) {
        const int g = q / sbb, sp = q - g * sbb;
        const int c0 = nb < 46341 ? sp * nb / sbb : (int)((long)sp * nb / sbb);
        const int c1 = nb < 46341 ? (sp + 1) * nb / sbb : (int)((long)(sp + 1) * nb / sbb);
        work[pos + q] = AttnWork{b, g, sp, sbb, c0, c1, c != raw ? ~c : c, slot + g * sbb};
      }
    }
  };
  // Up to 64 sequences: one wave sizes the list with shuffles (the same
  // integer steps as the block-wide path below, so the same list) and hands
  // each sequence's first slot and context to the writers.
  if (B <= kWave && B <= NT / 2) {
    if (wave == 0) {
      const int raw = lane < B ? ctx[lane] : 0;
      const unsigned n = lane < B ? (unsigned)nblocks_raw(raw) : 0u;
      const long total = wsum((int)n);
      const int pairs = B * Hkv;
      const long work_blocks = (long)Hkv * total;
      const int s_lo = max(kMinSplitBlocks, (int)((work_blocks + nwg - 1) / nwg));
      const int s_hi = nwg > pairs ? max(s_lo, (int)((work_blocks + (nwg - pairs) - 1) / (nwg - pairs))) : (1 << 28);
      int S = s_hi;
      for (int c = kCand - 1; c >= 0; --c) {
        const int cand = s_lo + (int)(((long)(s_hi - s_lo) * c + kCand - 2) / (kCand - 1));
        const int cnt = wsum(lane < B ? (int)max(1u, (n + (unsigned)cand - 1u) / (unsigned)cand) : 0);
        if ((long)cnt * Hkv <= nwg) S = cand;
      }
      const int items = lane < B ? Hkv * max(1, ((int)n + S - 1) / S) : 0;
      int incl = items;
      for (int o = 1; o < 64; o <<= 1) {
        const int up = __shfl_up(incl, o);
        if (lane >= o) incl += up;
      }
      if (lane < B) {
        s_seq[3 * lane] = incl - items;
        s_seq[3 * lane + 1] = raw;
      }
      if (lane == 63) {
        s_red[0] = S;
        s_red[1] = incl;
      }
    }
    __syncthreads();
    const int S = s_red[0], n_items = s_red[1];
    put_small(S);
    for (int i = n_items + threadIdx.x; i < nwg; i += NT) work[i] = AttnWork{};
    __syncthreads();  // scratch is free again
    return;
  }
  int keep[kKeep];
#pragma unroll
  for (int j = 0; j < kKeep; ++j) keep[j] = b0 + j < b1 ? ctx[b0 + j] : 0;
  auto raw_of = [&](int b) {
    const int i = b - b0;
    int r = 0;
#pragma unroll
    for (int j = 0; j < kKeep; ++j)
      if (i == j) r = keep[j];
    return i < kKeep ? r : ctx[b];
  };
  // sum of cached blocks
  int mine = 0;
  for (int b = b0; b < b1; ++b) mine += nblocks_raw(raw_of(b));
  mine = wsum(mine);
  __syncthreads();
  if (lane == 0) s_red[wave] = mine;
  __syncthreads();
  long total = 0;
  for (int w = 0; w < NWV; ++w) total += s_red[w];
  const int pairs = B * Hkv;
  const long work_blocks = (long)Hkv * total;
  const int s_lo = max(kMinSplitBlocks, (int)((work_blocks + nwg - 1) / nwg));
  const int s_hi = nwg > pairs ? max(s_lo, (int)((work_blocks + (nwg - pairs) - 1) / (nwg - pairs))) : (1 << 28);
  int cand[kCand], cnt[kCand];
#pragma unroll
  for (int c = 0; c < kCand; ++c) {
    cand[c] = s_lo + (int)(((long)(s_hi - s_lo) * c + kCand - 2) / (kCand - 1));
    cnt[c] = 0;
  }
  for (int b = b0; b < b1; ++b) {
    const unsigned n = (unsigned)nblocks_raw(raw_of(b));
#pragma unroll
    for (int c = 0; c < kCand; ++c) cnt[c] += max(1u, (n + (unsigned)cand[c] - 1u) / (unsigned)cand[c]);
  }
#pragma unroll
  for (int c = 0; c < kCand; ++c) cnt[c] = wsum(cnt[c]);
  __syncthreads();  // the block sums above are read
  if (lane == 0)
#pragma unroll
    for (int c = 0; c < kCand; ++c) s_red[wave * kCand + c] = cnt[c];
  __syncthreads();
  int S = s_hi;
#pragma unroll
  for (int c = kCand - 1; c >= 0; --c) {
    long items = 0;
    for (int w = 0; w < NWV; ++w) items += s_red[w * kCand + c];
    if (items * Hkv <= nwg) S = cand[c];
  }
  // exclusive scan of the per-thread item counts (threads own consecutive sequences)
  int my_items = 0;
  for (int b = b0; b < b1; ++b) my_items += Hkv * max(1, (nblocks_raw(raw_of(b)) + S - 1) / S);
  int incl = my_items;
  for (int o = 1; o < 64; o <<= 1) {
    const int up = __shfl_up(incl, o);
    if (lane >= o) incl += up;
  }
  __syncthreads();  // the candidate sums are read
  if (lane == 63) s_red[wave] = incl;
  __syncthreads();
  int start = incl - my_items, n_items = 0;
  for (int w = 0; w < NWV; ++w) {
    if (w < wave) start += s_red[w];
    n_items += s_red[w];
  }
  // the items: item q of sequence b (q = kv head * s_b + split) has partial
  // slot start_b + q and goes to the list position its split length gives.
  if (B <= NT / 2) {
    if ((int)threadIdx.x < B) {  // per == 1 here
      s_seq[3 * threadIdx.x] = start;
      s_seq[3 * threadIdx.x + 1] = keep[0];
    }
    __syncthreads();
    put_small(S);
  } else {
    if (order) {
      for (int i = threadIdx.x; i < kOrderBuckets; i += NT) s_hist[i] = 0;
      __syncthreads();
      for (int b = b0; b < b1; ++b) {
        const int n = nblocks_raw(raw_of(b)), sb = max(1, (n + S - 1) / S);
        atomicAdd(&s_hist[bucket(n, sb)], Hkv * sb);
      }
      scan_hist();
    }
    for (int b = b0; b < b1; ++b) {
      const int raw = raw_of(b);
      const int c = attn_clamp_ctx(raw, max_blocks, T), n = (c + kBlock - 1) / kBlock;
      const int sb = max(1, (n + S - 1) / S);
      const int pos = order ? atomicAdd(&s_hist[bucket(n, sb)], Hkv * sb) : start;
      for (int q = 0; q < Hkv * sb; ++q) {
        const int g = q / sb, sp = q - g * sb;
        const int c0 = n < 46341 ? sp * n / sb : (int)((long)sp * n / sb);
        const int c1 = n < 46341 ? (sp + 1) * n / sb : (int)((long)(sp + 1) * n / sb);
        work[pos + q] = AttnWork{b, g, sp, sb, c0, c1, c != raw ? ~c : c, start + g * sb};
      }
      start += Hkv * sb;
    }
  }
  for (int i = n_items + threadIdx.x; i < nwg; i += NT) work[i] = AttnWork{};
  __syncthreads();  // scratch is free again
}

// The arguments of a work-list build riding along another kernel's launch.
struct AttnPlan {
  const int32_t* ctx;
  AttnWork* work;  // nullptr: no build
  int B, Hkv, T, max_blocks, nwg;
  int order;       // longest splits first (attention_orders(nwg))
};

}  // namespace nj
