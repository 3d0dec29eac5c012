// Acceptance test of speculative sampling on the target logits.
//
// The test for draft i only needs p_i(x_i) and q_i(x_i), so all k tests are
// independent; the accepted length n is the index of the first failure.  The
// draw after it needs a running sum over one full vocabulary row, which is
// where the bandwidth goes.  Three kernels:
//
//   accept_stats   (rows x 8192-wide chunks): chunk max and sum of exp(l - max).
//   accept_tiles   (sequences x tile blocks): every workgroup first runs the
//                  k accept tests of its sequence (u_i < p_i(x_i) / q_i(x_i),
//                  q == 0 accepts; p from the chunk statistics) to find n, the
//                  first failure, then sums the draw weights of row n only --
//                  max(0, p_n - q_n) after a rejection, p_k for the bonus -- in
//                  fp64 over 256-wide tiles.  The tests are cheap and
//                  identical in every workgroup of a sequence.
//   accept_finalize (one wave per sequence): the smallest j whose running sum
//                  of row n's weights exceeds u_k times their total: a prefix
//                  scan over lane-contiguous tile sums finds the tile, a prefix
//                  scan over that tile's 256 weights finds the entry.  All sums
//                  are fp64 in a fixed order, so the draw is reproducible.
#include "common.h"
#include "kernels.h"

namespace nj {
namespace {

constexpr int kChunk = 8192;
constexpr int kStatThreads = 256;
constexpr int kTile = 256;          // weights per tile (4 per lane of a wave)
constexpr int kTilesPerBlock = 8;   // tiles per accept_tiles workgroup (two per wave)
constexpr int kMaxTiles = 2048;     // V <= 524288

// One pass: each thread holds its 32 values of the chunk in registers.
__global__ __launch_bounds__(kStatThreads) void accept_stats_kernel(const float* __restrict__ logits, int V, int nch,
                                                                    float* __restrict__ stats) {
  constexpr int PER = kChunk / kStatThreads / 4;  // float4 groups per thread
  __shared__ float sh[kStatThreads / kWave];
  const int row = blockIdx.x, c = blockIdx.y;
  const float* x = logits + (size_t)row * V;
  const int lo = c * kChunk, hi = min(lo + kChunk, V);
  float v[PER][4];
  float mx = -INFINITY;
  if ((V & 3) == 0) {
#pragma unroll
    for (int it = 0; it < PER; ++it) {
      const int j = lo + (it * kStatThreads + threadIdx.x) * 4;
      const f32x4 q = j < hi ? *reinterpret_cast<const f32x4*>(x + j) : f32x4{-INFINITY, -INFINITY, -INFINITY, -INFINITY};
#pragma unroll
      for (int e = 0; e < 4; ++e) v[it][e] = q[e];
    }
  } else {
#pragma unroll
    for (int it = 0; it < PER; ++it)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int j = lo + (it * kStatThreads + threadIdx.x) * 4 + e;
        v[it][e] = j < hi ? x[j] : -INFINITY;
      }
  }
#pragma unroll
  for (int it = 0; it < PER; ++it)
#pragma unroll
    for (int e = 0; e < 4; ++e) mx = fmaxf(mx, v[it][e]);
  mx = block_max<kStatThreads>(mx, sh);
  float s = 0.f;
#pragma unroll
  for (int it = 0; it < PER; ++it)
#pragma unroll
    for (int e = 0; e < 4; ++e) s += (v[it][e] == -INFINITY) ? 0.f : expf(v[it][e] - mx);
  s = block_sum<kStatThreads>(s, sh);
  if (threadIdx.x == 0) {
    stats[((size_t)row * nch + c) * 2] = mx;
    stats[((size_t)row * nch + c) * 2 + 1] = s;
  }
}

// Row max and 1/sum from the chunk statistics, in chunk order.
__device__ __forceinline__ void row_stats(const float* __restrict__ st, int nch, float* m, float* inv_s) {
  float mx = -INFINITY;
  for (int c = 0; c < nch; ++c) mx = fmaxf(mx, st[2 * c]);
  float s = 0.f;
  for (int c = 0; c < nch; ++c) s += st[2 * c + 1] * expf(st[2 * c] - mx);
  *m = mx;
  *inv_s = 1.0f / s;
}

// Weight of vocabulary entry j in a draw row: p_j, or max(0, p_j - q_j).
__device__ __forceinline__ float draw_weight(const float* __restrict__ lrow, const float* __restrict__ qrow,
                                             float m, float inv_s, bool resid, int j) {
  const float p = expf(lrow[j] - m) * inv_s;
  return resid ? fmaxf(0.f, p - qrow[j]) : p;
}

struct AccK {
  const float* logits;    // [B*T][V]
  const int32_t* drafts;  // [B][k]
  const float* dprobs;    // [B][k][V]
  const float* uniforms;  // [B][T]
  const float* stats;     // [B*T][nch][2]
  float* rowstat;         // [B][2]: max, 1/sum of the draw row
  double* tsum;           // [B][ntile]: tile sums of the draw row
  int32_t* nsel;          // [B]: accepted length n
  int32_t* accepted_len;
  int32_t* next_tokens;
  int* err;
  int k, V, nch, ntile;
};

__global__ __launch_bounds__(256) void accept_tiles_kernel(AccK a) {
  __shared__ float s_m[kWave], s_inv[kWave];
  __shared__ int s_n;
  const int b = blockIdx.x, T = a.k + 1, V = a.V;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (wave == 0) {
    // row statistics of the window rows (lane i: row i) and the k accept tests
    float m = 0.f, inv_s = 0.f;
    if (lane < T) {
      row_stats(a.stats + (size_t)(b * T + lane) * a.nch * 2, a.nch, &m, &inv_s);
      s_m[lane] = m;
      s_inv[lane] = inv_s;
    }
    bool ok = true;
    if (lane < a.k) {
      const int x = a.drafts[b * a.k + lane];
      if (x < 0 || x >= V) {
        if (blockIdx.y == 0) flag_error(a.err, kErrToken);
        ok = false;
      } else {
        const float p = expf(a.logits[(size_t)(b * T + lane) * V + x] - m) * inv_s;
        const float q = a.dprobs[((size_t)b * a.k + lane) * V + x];
        ok = (q <= 0.f) || (a.uniforms[b * T + lane] < p / q);
      }
    }
    const unsigned long long fails = __ballot(lane < a.k && !ok);
    const int n = fails ? __ffsll((long long)fails) - 1 : a.k;
    if (lane == 0) {
      s_n = n;
      if (blockIdx.y == 0) a.nsel[b] = n;
    }
  }
  __syncthreads();
  const int n = s_n;
  const float m = s_m[n], inv_s = s_inv[n];
  if (blockIdx.y == 0 && threadIdx.x == 0) {
    a.rowstat[b * 2] = m;
    a.rowstat[b * 2 + 1] = inv_s;
  }
  const bool resid = n < a.k;
  const float* lrow = a.logits + (size_t)(b * T + n) * V;
  const float* qrow = resid ? a.dprobs + ((size_t)b * a.k + n) * V : lrow;
  const int t0 = blockIdx.y * kTilesPerBlock, t1 = min(t0 + kTilesPerBlock, a.ntile);
  const bool vec = (a.V & 3) == 0;
  for (int t = t0 + wave; t < t1; t += 4) {
    const int j0 = t * kTile + lane * 4;
    double ls = 0.0;
    if (vec && j0 + 3 < a.V) {
      const f32x4 l4 = *reinterpret_cast<const f32x4*>(lrow + j0);
      const f32x4 q4 = *reinterpret_cast<const f32x4*>(qrow + j0);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float p = expf(l4[e] - m) * inv_s;
        ls += (double)(resid ? fmaxf(0.f, p - q4[e]) : p);
      }
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (j0 + e < a.V) ls += (double)draw_weight(lrow, qrow, m, inv_s, resid, j0 + e);
    }
    ls = wave_sum_d(ls);
    if (lane == 0) a.tsum[(size_t)b * a.ntile + t] = ls;
  }
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

__global__ __launch_bounds__(64) void accept_finalize_kernel(AccK a) {
  __shared__ double fb_tsum[kMaxTiles];  // only for an all-zero residual
  const int b = blockIdx.x, T = a.k + 1, V = a.V, lane = threadIdx.x;

  const int n = a.nsel[b];
  const int row = b * T + n;
  bool resid = n < a.k;
  const float* lrow = a.logits + (size_t)row * V;
  const float* qrow = resid ? a.dprobs + ((size_t)b * a.k + n) * V : lrow;
  const float m = a.rowstat[b * 2], inv_s = a.rowstat[b * 2 + 1];
  const int ntile = a.ntile;
  const double* ts = a.tsum + (size_t)b * ntile;

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
    __syncthreads();
    ts = fb_tsum;
    ls = 0.0;
    for (int t = t0; t < t1; ++t) ls += ts[t];
    incl = wave_incl_scan(ls);
    total = __shfl(incl, kWave - 1);
  }
  const double target = (double)a.uniforms[b * T + a.k] * total;

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
    if (lane < n) v = a.drafts[b * a.k + lane];
    else if (lane == n) v = cand;
    a.next_tokens[b * T + lane] = v;
  }
  if (lane == 0) a.accepted_len[b] = n;
}

size_t al256(size_t x) { return (x + 255) & ~(size_t)255; }

}  // namespace

int accept_chunks(int V) { return (V + kChunk - 1) / kChunk; }

size_t accept_workspace_bytes(int rows, int V) {
  const int ntile = (V + kTile - 1) / kTile;
  return al256((size_t)rows * accept_chunks(V) * 2 * 4) + al256((size_t)rows * 2 * 4) +
         al256((size_t)rows * ntile * 8) + al256((size_t)rows * 4);
}

hipError_t launch_accept(const AcceptArgs& x, hipStream_t s) {
  const int T = x.k + 1, rows = x.B * T, nch = accept_chunks(x.V), ntile = (x.V + kTile - 1) / kTile;
  char* ws = static_cast<char*>(x.scratch);
  float* stats = reinterpret_cast<float*>(ws);
  float* rowstat = reinterpret_cast<float*>(ws + al256((size_t)rows * nch * 2 * 4));
  double* tsum = reinterpret_cast<double*>(ws + al256((size_t)rows * nch * 2 * 4) + al256((size_t)rows * 2 * 4));
  int32_t* nsel = reinterpret_cast<int32_t*>(ws + al256((size_t)rows * nch * 2 * 4) + al256((size_t)rows * 2 * 4) +
                                             al256((size_t)rows * ntile * 8));
  hipLaunchKernelGGL(accept_stats_kernel, dim3(rows, nch), dim3(kStatThreads), 0, s, x.logits, x.V, nch, stats);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  AccK a{x.logits, x.drafts, x.dprobs, x.uniforms, stats, rowstat, tsum, nsel, x.accepted_len, x.next_tokens,
         x.err, x.k, x.V, nch, ntile};
  hipLaunchKernelGGL(accept_tiles_kernel, dim3(x.B, (ntile + kTilesPerBlock - 1) / kTilesPerBlock), dim3(256), 0,
                     s, a);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(accept_finalize_kernel, dim3(x.B), dim3(64), 0, s, a);
  return hipGetLastError();
}

}  // namespace nj
