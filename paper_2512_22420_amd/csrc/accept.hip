// Acceptance test of speculative sampling on the target logits.
//
// The test for draft i only needs p_i(x_i) and q_i(x_i), so all k tests are
// independent; the accepted length n is the index of the first failure.  The
// draw after it needs a running sum over one full vocabulary row, which is
// where the bandwidth goes.
//
//   statistics        (max, sum of exp(l - max)) pairs of every window row
//                     over disjoint column sets.  The LM-head GEMM writes them
//                     from its output tiles (one pair per workgroup and row,
//                     its 128-wide chunks merged; chunk_stats is shared);
//                     accept_stats_kernel computes one pair per 128-wide
//                     chunk from logits in memory when the GEMM did not.
//   accept_rows       (one workgroup per window row): row max and 1/sum from
//                     the statistics pairs, and the accept test of the draft
//                     the row scores (u_i < p_i(x_i) / q_i(x_i); q == 0
//                     accepts).
//   accept_draw       (sequences x tile blocks): n, the first failed test, then
//                     fp64 sums of the draw weights
//                     of row n over 256-wide tiles -- max(0, p_n - q_n) after
//                     a rejection, p_k for the bonus -- and the last workgroup
//                     of a sequence to finish (device-scope counter) draws:
//                     the smallest j whose running sum of row n's weights
//                     exceeds u_k times their total, found by a prefix scan
//                     over lane-contiguous tile sums and one over the chosen
//                     tile's 256 weights.  All sums are fp64 in a fixed order,
//                     so the draw is reproducible.
#include "common.h"
#include "kernels.h"

namespace nj {
namespace {

constexpr int kTile = 256;          // weights per tile (4 per lane of a wave)
// Tiles a wave of accept_draw sums (its loads issued together): two while few
// sequences leave the grid small, four from kDrawWideBatch sequences up
// (fewer, longer workgroups: B=128 at the 8B vocabulary 53 -> 48 us, B=256
// at the 7B vocabulary 109 -> 87 us; at B=8 two are faster).
constexpr int kDrawWideBatch = 32;
constexpr int kMaxTiles = 2048;     // V <= 524288

struct AccK {
  const float* logits;    // [B*T][V]
  const int32_t* drafts;  // [B][k]
  const float* dprobs;    // [B][k][V]
  const float* uniforms;  // [B][T]
  const float* stats;     // [B*T][nch][2]; entries 0 .. nst-1 of each row are used
  float* rowstat;         // [B*T][2]: max, 1/sum of every window row
  int32_t* okflag;        // [B*T]: accept test of the draft row i scores (rows 0..k-1)
  double* tsum;           // [B][ntile]: tile sums of the draw row
  int* counters;          // [B][kCounterStride]: draw arrivals (zeroed by accept_rows)
  int32_t* accepted_len;
  int32_t* next_tokens;
  int* err;
  int k, V, nch, nst, ntile, tsum_bytes;
};

// 128-wide chunks of the logits, written by 256-thread workgroups (8 lanes per chunk).
__global__ __launch_bounds__(256) void accept_stats_kernel(const float* __restrict__ logits, int V, int nch,
                                                           float* __restrict__ stats) {
  const int row = blockIdx.x;
  const int chunk = blockIdx.y * 32 + threadIdx.x / kStatLanes, c = threadIdx.x % kStatLanes;
  const int cc = min(chunk, nch - 1);  // surplus lanes of the last block repeat the last chunk (not stored)
  const float* x = logits + (size_t)row * V;
  float v[kStatPer];
  const int j0 = cc * kStatChunk + c * kStatPer;
#pragma unroll
  for (int e = 0; e < kStatPer; ++e) v[e] = j0 + e < V ? x[j0 + e] : -INFINITY;
  float m, sum;
  chunk_stats(v, m, sum);
  if (c == 0 && chunk < nch) {
    stats[((size_t)row * nch + chunk) * 2] = m;
    stats[((size_t)row * nch + chunk) * 2 + 1] = sum;
  }
}

// One workgroup per window row: the row max and 1/sum from the chunk
// statistics (thread t takes chunks t, t+256, ...; all its loads are issued
// before any is used), and, for rows 0..k-1, the accept test of the draft the
// row scores.  Row 0 of each sequence also clears the sequence's draw counter.
constexpr int kRowThreads = 256, kRowLoads = 16;  // chunks per thread (V <= 524288)
__global__ __launch_bounds__(kRowThreads) void accept_rows_kernel(AccK a) {
  __shared__ float sh[kRowThreads / kWave];
  const int row = blockIdx.x, T = a.k + 1, b = row / T, i = row % T, V = a.V, nst = a.nst;
  const float* st = a.stats + (size_t)row * a.nch * 2;
  // the draft this row scores, and its target logit and draft probability
  float lx = 0.f, qx = 1.f;
  bool bad = false;
  if (threadIdx.x == 0 && i < a.k) {
    const int x = a.drafts[b * a.k + i];
    bad = x < 0 || x >= V;
    const int xs = bad ? 0 : x;
    lx = a.logits[(size_t)row * V + xs];
    qx = a.dprobs[((size_t)b * a.k + i) * V + xs];
  }
  float cm[kRowLoads], cs[kRowLoads];
#pragma unroll
  for (int j = 0; j < kRowLoads; ++j) {
    const int c = threadIdx.x + j * kRowThreads;
    const int cc = min(c, nst - 1);
    cm[j] = c < nst ? st[2 * cc] : -INFINITY;
    cs[j] = c < nst ? st[2 * cc + 1] : 0.f;
  }
  float m = cm[0];
#pragma unroll
  for (int j = 1; j < kRowLoads; ++j) m = fmaxf(m, cm[j]);
  m = block_max<kRowThreads>(m, sh);
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < kRowLoads; ++j) s += (cm[j] == -INFINITY) ? 0.f : cs[j] * expf(cm[j] - m);
  s = block_sum<kRowThreads>(s, sh);
  if (threadIdx.x == 0) {
    const float inv_s = 1.0f / s;
    a.rowstat[row * 2] = m;
    a.rowstat[row * 2 + 1] = inv_s;
    if (i < a.k) {
      if (bad) flag_error(a.err, kErrToken);
      const float p = expf(lx - m) * inv_s;
      a.okflag[row] = !bad && ((qx <= 0.f) || (a.uniforms[row] < p / qx));
    }
    if (i == 0) a.counters[b * kCounterStride] = 0;
  }
}

// Weight of vocabulary entry j in a draw row: p_j, or max(0, p_j - q_j).
__device__ __forceinline__ float draw_weight(const float* __restrict__ lrow, const float* __restrict__ qrow,
                                             float m, float inv_s, bool resid, int j) {
  const float p = expf(lrow[j] - m) * inv_s;
  return resid ? fmaxf(0.f, p - qrow[j]) : p;
}

// Inclusive prefix sum over the 64 lanes of a wave.
__device__ __forceinline__ double wave_incl_scan(double v) {
  const int lane = threadIdx.x & 63;
  for (int o = 1; o < kWave; o <<= 1) {
    const double up = __shfl_up(v, o);
    if (lane >= o) v += up;
  }
  return v;
}

// The draw of sequence b from its tile sums ts[0..ntile) (LDS), run by one wave.
// u: the draw's uniform; dft: draft `lane` of the sequence (lanes < k).
__device__ void draw_token(const AccK& a, int b, int n, bool resid, float m, float inv_s, float u, int dft, double* ts,
                           double* fb_tsum) {
  const int T = a.k + 1, V = a.V, lane = threadIdx.x & 63;
  const int row = b * T + n;
  const float* lrow = a.logits + (size_t)row * V;
  const float* qrow = resid ? a.dprobs + ((size_t)b * a.k + n) * V : lrow;
  const int ntile = a.ntile;

  // lane-contiguous tile ranges; the total is the last inclusive prefix, so it
  // is made of exactly the additions the search below walks through
  const int per = (ntile + kWave - 1) / kWave;
  const int t0 = min(lane * per, ntile), t1 = min(t0 + per, ntile);
  double ls = 0.0;
  for (int t = t0; t < t1; ++t) ls += ts[t];
  double incl = wave_incl_scan(ls);
  double total = __shfl(incl, kWave - 1);
  if (resid && !(total > 0.0)) {
    // max(0, p_n - q_n) vanished (only rounding can do that): draw from p_n
    resid = false;
    qrow = lrow;
    for (int t = 0; t < ntile; ++t) {
      double s = 0.0;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int j = t * kTile + lane * 4 + e;
        if (j < V) s += (double)draw_weight(lrow, qrow, m, inv_s, false, j);
      }
      s = wave_sum_d(s);
      if (lane == 0) fb_tsum[t] = s;
    }
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    ts = fb_tsum;
    ls = 0.0;
    for (int t = t0; t < t1; ++t) ls += ts[t];
    incl = wave_incl_scan(ls);
    total = __shfl(incl, kWave - 1);
  }
  const double target = (double)u * total;

  int tile = -1;
  double base = 0.0;
  int want_last = 0;  // take the last positive entry of `tile` instead of searching
  const unsigned long long hit = __ballot(incl > target);
  if (hit) {
    const int L = __ffsll((long long)hit) - 1;
    if (lane == L) {
      double cum = incl - ls;
      for (int t = t0; t < t1; ++t) {
        if (cum + ts[t] > target) {
          tile = t;
          base = cum;
          break;
        }
        cum += ts[t];
      }
      if (tile < 0) {  // rounding: the last positive tile of this lane's range
        for (int t = t1 - 1; t >= t0; --t)
          if (ts[t] > 0.0) {
            tile = t;
            break;
          }
        want_last = 1;
      }
    }
    tile = __shfl(tile, L);
    base = __shfl(base, L);
    want_last = __shfl(want_last, L);
  } else {
    // no running sum exceeds u*S (u close to 1): the last positive weight
    int tl = -1;
    for (int t = ntile - 1 - lane; t >= 0; t -= kWave)
      if (ts[t] > 0.0) {
        tl = t;
        break;
      }
    for (int o = 32; o > 0; o >>= 1) tl = max(tl, __shfl_xor(tl, o));
    tile = tl;
    want_last = 1;
  }
  if (tile < 0) tile = 0;

  float w4[4];
  double lsum = 0.0;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int j = tile * kTile + lane * 4 + e;
    w4[e] = (j < V) ? draw_weight(lrow, qrow, m, inv_s, resid, j) : 0.f;
    lsum += (double)w4[e];
  }
  int cand = -1;
  if (!want_last) {
    const double inc = wave_incl_scan(lsum);
    const unsigned long long h2 = __ballot(base + inc > target);
    if (h2) {
      const int L = __ffsll((long long)h2) - 1;
      if (lane == L) {
        double cum = base + inc - lsum;
        for (int e = 0; e < 4; ++e) {
          cum += (double)w4[e];
          if (w4[e] > 0.f && cum > target) {
            cand = tile * kTile + lane * 4 + e;
            break;
          }
        }
      }
    }
    for (int o = 32; o > 0; o >>= 1) cand = max(cand, __shfl_xor(cand, o));
  }
  if (cand < 0) {
    int lastpos = -1;
#pragma unroll
    for (int e = 0; e < 4; ++e)
      if (w4[e] > 0.f) lastpos = tile * kTile + lane * 4 + e;
    for (int o = 32; o > 0; o >>= 1) lastpos = max(lastpos, __shfl_xor(lastpos, o));
    cand = lastpos < 0 ? tile * kTile : lastpos;
  }

  if (lane < T) {
    int v = -1;
    if (lane < n) v = dft;
    else if (lane == n) v = cand;
    a.next_tokens[b * T + lane] = v;
  }
  if (lane == 0) a.accepted_len[b] = n;
}

template <int kTilesPerWave>
__global__ __launch_bounds__(256) void accept_draw_kernel(AccK a) {
  constexpr int kTilesPerBlock = 4 * kTilesPerWave;
  __shared__ double s_ts[kMaxTiles];
  __shared__ double s_fb[kMaxTiles];  // only for an all-zero residual
  __shared__ int s_last;
  const int b = blockIdx.x, T = a.k + 1;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  // n = index of the first failed test (k if all passed); the test flags, the
  // statistics of every window row, the draw's uniform and the drafts are
  // loaded together, before anything depends on n
  int okv = 1, dft = -1;
  float rm = 0.f, ri = 0.f;
  if (lane < a.k) {
    okv = a.okflag[b * T + lane];
    dft = a.drafts[b * a.k + lane];
  }
  if (lane < T) {
    rm = a.rowstat[(b * T + lane) * 2];
    ri = a.rowstat[(b * T + lane) * 2 + 1];
  }
  const float u = a.uniforms[b * T + a.k];
  const unsigned long long fails = __ballot(lane < a.k && !okv);
  const int n = fails ? __ffsll((long long)fails) - 1 : a.k;
  const float m = __shfl(rm, n), inv_s = __shfl(ri, n);
  const bool resid = n < a.k;
  const float* lrow = a.logits + (size_t)(b * T + n) * a.V;
  const float* qrow = resid ? a.dprobs + ((size_t)b * a.k + n) * a.V : lrow;
  const __amdgpu_buffer_rsrc_t trs = coherent_rsrc(a.tsum, a.tsum_bytes);
  // this wave's tiles t0 + wave + 4 j: every tile's loads are issued before
  // any is summed (whole vec4 pieces; the row's ragged end takes the scalar path)
  const int t0 = blockIdx.y * kTilesPerBlock;
  const bool vec = (a.V & 3) == 0;
  f32x4 l4[kTilesPerWave], q4[kTilesPerWave];
#pragma unroll
  for (int j = 0; j < kTilesPerWave; ++j) {
    const int t = t0 + wave + 4 * j, j0 = t * kTile + lane * 4;
    const bool full = vec && t < a.ntile && j0 + 3 < a.V;
    l4[j] = full ? *reinterpret_cast<const f32x4*>(lrow + j0) : f32x4{0.f, 0.f, 0.f, 0.f};
    q4[j] = full && resid ? *reinterpret_cast<const f32x4*>(qrow + j0) : f32x4{0.f, 0.f, 0.f, 0.f};
  }
#pragma unroll
  for (int j = 0; j < kTilesPerWave; ++j) {
    const int t = t0 + wave + 4 * j;
    if (t >= a.ntile) break;
    const int j0 = t * kTile + lane * 4;
    double ls = 0.0;
    if (vec && j0 + 3 < a.V) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float p = expf(l4[j][e] - m) * inv_s;
        ls += (double)(resid ? fmaxf(0.f, p - q4[j][e]) : p);
      }
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (j0 + e < a.V) ls += (double)draw_weight(lrow, qrow, m, inv_s, resid, j0 + e);
    }
    ls = wave_sum_d(ls);
    if (lane == 0) coherent_store_f64(trs, (uint32_t)(((size_t)b * a.ntile + t) * 8), ls);
  }
  // the last workgroup of the sequence to arrive draws (tile sums written and
  // read with device-coherent accesses, published by the counter increment)
  __asm__ volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  if (threadIdx.x == 0)
    s_last = (__hip_atomic_fetch_add(a.counters + b * kCounterStride, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
              (int)gridDim.y - 1);
  __syncthreads();
  if (!s_last) return;
  for (int t = threadIdx.x; t < a.ntile; t += 256)
    s_ts[t] = coherent_load_f64(trs, (uint32_t)(((size_t)b * a.ntile + t) * 8));
  __syncthreads();
  if (wave == 0) draw_token(a, b, n, resid, m, inv_s, u, dft, s_ts, s_fb);
}

size_t al256(size_t x) { return (x + 255) & ~(size_t)255; }

// A draft step (k = 0): sequence b's drawn token goes to tokens[b * tstride]
// and its distribution p_j = exp(l_j - m) / sum to probs[b * pstride + j],
// from the row statistics accept_rows wrote (the same fp32 values the draw
// summed).  grid (B, ceil(V / 1024)), 4 entries per thread.
__global__ __launch_bounds__(256) void emit_draft_kernel(const float* __restrict__ logits,
                                                         const float* __restrict__ rowstat,
                                                         const int32_t* __restrict__ next, int V,
                                                         int32_t* __restrict__ tokens, int tstride,
                                                         float* __restrict__ probs, long long pstride) {
  const int b = blockIdx.x;
  const float m = rowstat[b * 2], inv_s = rowstat[b * 2 + 1];
  if (blockIdx.y == 0 && threadIdx.x == 0) tokens[(size_t)b * tstride] = next[b];
  const float* l = logits + (size_t)b * V;
  float* p = probs + (size_t)b * pstride;
  const int j0 = (blockIdx.y * 256 + threadIdx.x) * 4;
#pragma unroll
  for (int e = 0; e < 4; ++e)
    if (j0 + e < V) p[j0 + e] = expf(l[j0 + e] - m) * inv_s;
}

}  // namespace

int accept_chunks(int V) { return (V + kStatChunk - 1) / kStatChunk; }

// [stats][rowstat][tsum][okflag][counters]
size_t accept_workspace_bytes(int rows, int V) {
  const int ntile = (V + kTile - 1) / kTile;
  return al256((size_t)rows * accept_chunks(V) * 2 * 4) + al256((size_t)rows * 2 * 4) +
         al256((size_t)rows * ntile * 8) + al256((size_t)rows * 4) + al256((size_t)rows * kCounterStride * 4);
}

float* accept_stats_ptr(void* scratch) { return static_cast<float*>(scratch); }

hipError_t launch_emit_draft(const AcceptArgs& x, int32_t* tokens, int tstride, float* probs, long long pstride,
                             hipStream_t s) {
  if (x.k != 0) return hipErrorInvalidValue;
  const int rows = x.B, nch = accept_chunks(x.V);
  const float* rowstat = reinterpret_cast<const float*>(static_cast<char*>(x.scratch) + al256((size_t)rows * nch * 2 * 4));
  hipLaunchKernelGGL(emit_draft_kernel, dim3(x.B, (x.V + 1023) / 1024), dim3(256), 0, s, x.logits, rowstat,
                     x.next_tokens, x.V, tokens, tstride, probs, pstride);
  return hipGetLastError();
}

hipError_t launch_accept(const AcceptArgs& x, hipStream_t s) {
  const int T = x.k + 1, rows = x.B * T, nch = accept_chunks(x.V), ntile = (x.V + kTile - 1) / kTile;
  char* ws = static_cast<char*>(x.scratch);
  size_t off = 0;
  float* stats = reinterpret_cast<float*>(ws + off);
  off += al256((size_t)rows * nch * 2 * 4);
  float* rowstat = reinterpret_cast<float*>(ws + off);
  off += al256((size_t)rows * 2 * 4);
  double* tsum = reinterpret_cast<double*>(ws + off);
  const size_t tsum_bytes = (size_t)x.B * ntile * 8;
  off += al256((size_t)rows * ntile * 8);
  int32_t* okflag = reinterpret_cast<int32_t*>(ws + off);
  off += al256((size_t)rows * 4);
  int* counters = reinterpret_cast<int*>(ws + off);
  hipError_t e;
  if (!x.stats_ready) {
    hipLaunchKernelGGL(accept_stats_kernel, dim3(rows, (nch + 31) / 32), dim3(256), 0, s, x.logits, x.V, nch, stats);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  const int nst = x.stats_ready ? x.stat_entries : nch;
  if (nst < 1 || nst > nch || nst > kRowThreads * kRowLoads) return hipErrorInvalidValue;
  AccK a{x.logits, x.drafts, x.dprobs, x.uniforms, stats, rowstat, okflag, tsum, counters, x.accepted_len,
         x.next_tokens, x.err, x.k, x.V, nch, nst, ntile, (int)tsum_bytes};
  hipLaunchKernelGGL(accept_rows_kernel, dim3(rows), dim3(kRowThreads), 0, s, a);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (x.B >= kDrawWideBatch)
    hipLaunchKernelGGL(accept_draw_kernel<4>, dim3(x.B, (ntile + 15) / 16), dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL(accept_draw_kernel<2>, dim3(x.B, (ntile + 7) / 8), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace nj
