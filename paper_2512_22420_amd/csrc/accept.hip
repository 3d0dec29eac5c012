// Acceptance test of speculative sampling on the target logits.
//
// Stage 1 (accept_stats): per (window row, 8192-wide vocab chunk) the chunk
// max and the sum of exp(logit - max): the softmax normaliser of every row
// without a full-row pass in one workgroup.
//
// Stage 2 (accept_finalize): one workgroup of 16 waves per sequence.
//   - row statistics from the chunk partials (fixed order);
//   - the accept loop over drafts: x_i is accepted iff u_i < p_i(x_i)/q_i(x_i)
//     (q_i(x_i) == 0 accepts), stopping at the first rejection n;
//   - the weights of the final draw, w = max(0, p_n - q_n) after a rejection
//     (p_n if that is all zero) or w = p_k for the bonus token;
//   - the inverse CDF: the smallest j with sum_{i<=j} w_i > u_k * sum(w),
//     found by fp64 sums over 256-wide tiles (one per wave step), a wave
//     prefix scan over the tile sums to locate the tile, and a wave prefix
//     scan inside that tile.  Every sum is accumulated in fp64 in a fixed order,
//     so the draw is reproducible; against a sequential fp64 running sum of the
//     same fp32 weights only the summation order differs (~1e-15 relative).
#include "common.h"
#include "kernels.h"

namespace nj {
namespace {

constexpr int kChunk = 8192;
constexpr int kStatThreads = 256;
constexpr int kAccThreads = 1024;
constexpr int kAccWaves = kAccThreads / kWave;
constexpr int kTile = 256;       // elements per wave step (4 per lane)
constexpr int kMaxTiles = 2048;  // V <= 524288
constexpr int kMaxT = 16;

__global__ __launch_bounds__(kStatThreads) void accept_stats_kernel(const float* __restrict__ logits, int V, int nch,
                                                                    float* __restrict__ stats) {
  __shared__ float sh[kStatThreads / kWave];
  const int row = blockIdx.x, c = blockIdx.y;
  const float* x = logits + (size_t)row * V;
  const int lo = c * kChunk, hi = min(lo + kChunk, V);
  float mx = -INFINITY;
  for (int j = lo + threadIdx.x; j < hi; j += kStatThreads) mx = fmaxf(mx, x[j]);
  mx = block_max<kStatThreads>(mx, sh);
  float s = 0.f;
  for (int j = lo + threadIdx.x; j < hi; j += kStatThreads) s += expf(x[j] - mx);
  s = block_sum<kStatThreads>(s, sh);
  if (threadIdx.x == 0) {
    stats[((size_t)row * nch + c) * 2] = mx;
    stats[((size_t)row * nch + c) * 2 + 1] = s;
  }
}

struct AccK {
  const float* logits;
  const int32_t* drafts;
  const float* dprobs;
  const float* uniforms;
  const float* stats;
  int32_t* accepted_len;
  int32_t* next_tokens;
  int* err;
  int k, V, nch;
};

// weight of vocab entry j for the final draw
__device__ __forceinline__ float draw_weight(const float* __restrict__ lrow, const float* __restrict__ qrow,
                                             float m, float inv_s, bool resid, int j) {
  const float p = expf(lrow[j] - m) * inv_s;
  return resid ? fmaxf(0.f, p - qrow[j]) : p;
}

__global__ __launch_bounds__(kAccThreads) void accept_finalize_kernel(AccK a) {
  __shared__ float row_m[kMaxT], row_is[kMaxT];
  __shared__ double tsum[kMaxTiles];
  __shared__ int sh_n, sh_resid, sh_y;
  __shared__ double sh_total;

  const int b = blockIdx.x, T = a.k + 1, V = a.V;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;

  if (threadIdx.x < T) {
    const float* st = a.stats + (size_t)(b * T + threadIdx.x) * a.nch * 2;
    float mx = -INFINITY;
    for (int c = 0; c < a.nch; ++c) mx = fmaxf(mx, st[2 * c]);
    float s = 0.f;
    for (int c = 0; c < a.nch; ++c) s += st[2 * c + 1] * expf(st[2 * c] - mx);
    row_m[threadIdx.x] = mx;
    row_is[threadIdx.x] = 1.0f / s;
  }
  __syncthreads();

  if (threadIdx.x == 0) {
    int n = 0;
    for (; n < a.k; ++n) {
      const int x = a.drafts[b * a.k + n];
      if (x < 0 || x >= V) {
        flag_error(a.err, kErrToken);
        break;
      }
      const float p = expf(a.logits[(size_t)(b * T + n) * V + x] - row_m[n]) * row_is[n];
      const float q = a.dprobs[((size_t)b * a.k + n) * V + x];
      const bool acc = (q <= 0.f) || (a.uniforms[b * T + n] < p / q);
      if (!acc) break;
    }
    sh_n = n;
    sh_resid = n < a.k;
  }
  __syncthreads();

  const int n = sh_n;
  const float* lrow = a.logits + (size_t)(b * T + n) * V;
  // draft row of the rejected position (only read when there is a rejection)
  const float* qrow = (n < a.k) ? a.dprobs + ((size_t)b * a.k + n) * V : lrow;
  const float m = row_m[n], inv_s = row_is[n];
  const int ntile = (V + kTile - 1) / kTile;

  for (int pass = 0; pass < 2; ++pass) {
    const bool resid = sh_resid;
    for (int t = wave; t < ntile; t += kAccWaves) {
      double ls = 0.0;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int j = t * kTile + lane * 4 + e;
        if (j < V) ls += (double)draw_weight(lrow, qrow, m, inv_s, resid, j);
      }
      ls = wave_sum_d(ls);
      if (lane == 0) tsum[t] = ls;
    }
    __syncthreads();
    if (wave == 0) {
      double s = 0.0;
      for (int t = lane; t < ntile; t += kWave) s += tsum[t];
      s = wave_sum_d(s);
      if (lane == 0) {
        sh_total = s;
        // an all-zero residual (only rounding makes p_n <= q_n everywhere) falls back to p_n
        if (pass == 0 && resid && !(s > 0.0)) sh_resid = 0;
      }
    }
    __syncthreads();
    if (!(pass == 0 && resid && !sh_resid)) break;
  }

  if (wave == 0) {
    const bool resid = sh_resid;
    const double target = (double)a.uniforms[b * T + a.k] * sh_total;
    // contiguous tiles per lane, then a wave prefix scan over the lane sums
    const int per = (ntile + kWave - 1) / kWave;
    const int t0 = min(lane * per, ntile), t1 = min(t0 + per, ntile);
    double ls = 0.0;
    for (int t = t0; t < t1; ++t) ls += tsum[t];
    double incl = ls;
    for (int o = 1; o < kWave; o <<= 1) {
      const double up = __shfl_up(incl, o);
      if (lane >= o) incl += up;
    }
    const unsigned long long hit = __ballot(incl > target);
    int tile = -1;
    double base = 0.0;
    bool want_last = false;  // take the last positive entry of `tile` instead of searching
    if (hit) {
      const int L = __ffsll((long long)hit) - 1;
      if (lane == L) {
        double cum = incl - ls;
        for (int t = t0; t < t1; ++t) {
          if (cum + tsum[t] > target) {
            tile = t;
            base = cum;
            break;
          }
          cum += tsum[t];
        }
      }
      tile = __shfl(tile, L);
      base = __shfl(base, L);
      if (tile < 0) {
        // the lane-level and tile-level sums round differently and the target
        // fell between them: the last positive tile of lane L's range
        int tl = -1;
        if (lane == L)
          for (int t = t1 - 1; t >= t0; --t)
            if (tsum[t] > 0.0) {
              tl = t;
              break;
            }
        tile = __shfl(tl, L);
        want_last = true;
      }
    } else {
      // no running sum exceeds u*S (u close to 1): the last positive weight
      int tl = -1;
      for (int t = ntile - 1 - lane; t >= 0; t -= kWave)
        if (tsum[t] > 0.0) {
          tl = t;
          break;
        }
      for (int o = 32; o > 0; o >>= 1) tl = max(tl, __shfl_xor(tl, o));
      tile = tl;
      want_last = true;
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
      double inc = lsum;
      for (int o = 1; o < kWave; o <<= 1) {
        const double up = __shfl_up(inc, o);
        if (lane >= o) inc += up;
      }
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
    const int y = cand;
    if (lane == 0) sh_y = y;
  }
  __syncthreads();
  if (threadIdx.x < T) {
    const int t = threadIdx.x;
    int v = -1;
    if (t < n) v = a.drafts[b * a.k + t];
    else if (t == n) v = sh_y;
    a.next_tokens[b * T + t] = v;
  }
  if (threadIdx.x == 0) a.accepted_len[b] = n;
}

}  // namespace

int accept_chunks(int V) { return (V + kChunk - 1) / kChunk; }

hipError_t launch_accept(const AcceptArgs& x, hipStream_t s) {
  const int T = x.k + 1, nch = accept_chunks(x.V);
  hipLaunchKernelGGL(accept_stats_kernel, dim3(x.B * T, nch), dim3(kStatThreads), 0, s, x.logits, x.V, nch,
                     x.stats);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  AccK a{x.logits, x.drafts, x.dprobs, x.uniforms, x.stats, x.accepted_len, x.next_tokens, x.err, x.k, x.V, nch};
  hipLaunchKernelGGL(accept_finalize_kernel, dim3(x.B), dim3(kAccThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace nj
