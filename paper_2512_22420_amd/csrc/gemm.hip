// GEMMs of the verify step: y = x . w^T over the B*(k+1) window rows.
//
// bf16 path: weight-streaming MFMA kernel.  At verify-step sizes M = B*(k+1)
// is 1..~768 while N*K reaches 5e8 (LM head), so below M ~ 300 the work is
// bound by reading each weight byte once from HBM.
//
// - Each wave owns 16 weight rows -- the A operand of v_mfma_f32_16x16x32_bf16
//   -- and streams them along K with 16-byte loads, eight 32-wide k-steps per
//   stage, with the next stage's loads in flight while the current one is
//   multiplied (two register buffers, no copies between them).
// - The activation rows (B operand, M padded to 16) are staged per stage in
//   LDS, loaded once per workgroup and shared by all its waves (4 or 8), with
//   a 16-byte row pad against bank conflicts.  Reading them from L2 per wave
//   instead costs half the bandwidth at M = 48.
// - When 16-row tiles alone give too few workgroups to fill 256 CUs (small N),
//   K is split across workgroups: each writes an fp32 partial, and the last
//   workgroup of a tile to arrive (device-scope counter) adds the partials in
//   chunk order and applies the epilogue, so results do not depend on arrival
//   order.  Counters reset themselves for the next launch.
// - Epilogues: store fp32, add into the fp32 residual stream, or SwiGLU
//   (gate rows n and up rows Nout + n are two row groups of the same wave)
//   stored as bf16.
//
// Operand layout (16x16x32 bf16): lane l supplies row (l & 15) of A and
// column (l & 15) of B, eight consecutive k of k-group (l >> 4); the result
// lane l holds rows 4*(l >> 4) + i, column l & 15.  Any k permutation applied
// to both operands leaves the product unchanged.
#include <algorithm>
#include <cmath>

#include "common.h"
#include "kernels.h"

namespace nj {
namespace {

constexpr int kU = 8;                     // 32-wide k-steps per stage
constexpr int kStageK = 32 * kU;          // 256
constexpr int kRowStride = kStageK + 8;   // LDS row stride in elements (+16 bytes)
constexpr int kSplitTargetWorkgroups = 256;
// windows of at least this many rows may use the LDS-tiled kernel
constexpr int kTileMinRows = 64;

__device__ __forceinline__ bf16x8 ld8(const bf16_t* p) {
  return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(p));
}

__device__ __forceinline__ float silu_mul(float gte, float up) { return gte / (1.0f + expf(-gte)) * up; }

struct GemmK {
  const bf16_t* X;
  const bf16_t* W;
  void* Y;
  float* part;    // [nkc][M][NG][Nout] fp32 partials (split K only)
  int* counters;  // [mblocks][ntiles] arrival counters (split K only), zero between launches
  int M, Nout, K, stages_per_chunk;
  int part_bytes;
};

// MT: 16-row x tiles per workgroup; NG: weight row groups (2 for SwiGLU);
// NW: waves per workgroup (each owns 16 weight rows of every group).
// FULL: K % 256 == 0 and every wave owns 16 real weight rows, so the stage loop
// needs no guards at all; the prefetch of the stage after the last one simply
// re-reads the last one (an L1/L2 hit).  Branches inside the loop would make
// the compiler drain all outstanding loads at every join.
template <int MT, int NG, int NW, int EPI, int DEPTH, bool FULL>
__global__ __launch_bounds__(NW * 64) void gemm_bf16_kernel(GemmK a) {
  constexpr int ROWS = MT * 16, NTH = NW * 64;
  constexpr int CHUNKS = ROWS * kStageK / 8;  // 16-byte pieces of one x stage
  constexpr int PER_T = (CHUNKS + NTH - 1) / NTH;
  __shared__ __attribute__((aligned(16))) bf16_t xs[2][ROWS * kRowStride];
  __shared__ int s_last;

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r = lane & 15, g = lane >> 4;
  const int tile = blockIdx.x, mb = blockIdx.y, kc = blockIdx.z, nkc = gridDim.z;
  const int M = a.M, Nout = a.Nout, K = a.K;
  const int n0 = (tile * NW + wave) * 16;
  const int m0 = mb * ROWS;
  const bool active = n0 < Nout;
  const int S = K / 32;
  const int nst = (S + kU - 1) / kU;
  const int st0 = kc * a.stages_per_chunk, st1 = min(nst, st0 + a.stages_per_chunk);

  const int nrow = min(n0 + r, Nout - 1);
  const bf16_t* wp[NG];
#pragma unroll
  for (int q = 0; q < NG; ++q) wp[q] = a.W + (size_t)(q * Nout + nrow) * K + g * 8;

  f32x4 acc[MT][NG];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int q = 0; q < NG; ++q) acc[mt][q] = f32x4{0.f, 0.f, 0.f, 0.f};

  u32x4 xr[PER_T];
  bf16x8 wbuf[DEPTH + 1][NG][kU];

#define NJ_GLOAD_X(st)                                                                           \
  _Pragma("unroll") for (int c = 0; c < PER_T; ++c) {                                            \
    const int idx = threadIdx.x + c * NTH;                                                       \
    if (idx < CHUNKS) {                                                                          \
      const int row = idx / (kStageK / 8), kk = (st) * kStageK + (idx % (kStageK / 8)) * 8;      \
      xr[c] = kk < K ? *reinterpret_cast<const u32x4*>(a.X + (size_t)min(m0 + row, M - 1) * K + kk) \
                     : u32x4{0u, 0u, 0u, 0u};                                                    \
    }                                                                                            \
  }
#define NJ_SSTORE_X(buf)                                                                         \
  _Pragma("unroll") for (int c = 0; c < PER_T; ++c) {                                            \
    const int idx = threadIdx.x + c * NTH;                                                       \
    if (idx < CHUNKS) {                                                                          \
      const int row = idx / (kStageK / 8), col = (idx % (kStageK / 8)) * 8;                      \
      *reinterpret_cast<u32x4*>(&xs[buf][row * kRowStride + col]) = xr[c];                       \
    }                                                                                            \
  }
#define NJ_LOAD_W(B, st)                                                                         \
  if (active) {                                                                                  \
    _Pragma("unroll") for (int u = 0; u < kU; ++u) {                                             \
      if ((st) * kU + u < S) {                                                                   \
        _Pragma("unroll") for (int q = 0; q < NG; ++q) wbuf[B][q][u] = ld8(wp[q] + ((st) * kU + u) * 32); \
      }                                                                                          \
    }                                                                                            \
  }
#define NJ_COMPUTE(B, buf, st)                                                                   \
  if (active) {                                                                                  \
    _Pragma("unroll") for (int u = 0; u < kU; ++u) {                                             \
      if ((st) * kU + u < S) {                                                                   \
        _Pragma("unroll") for (int mt = 0; mt < MT; ++mt) {                                      \
          const bf16x8 xv = __builtin_bit_cast(                                                  \
              bf16x8, *reinterpret_cast<const u32x4*>(&xs[buf][(mt * 16 + r) * kRowStride + u * 32 + g * 8])); \
          _Pragma("unroll") for (int q = 0; q < NG; ++q) acc[mt][q] =                            \
              __builtin_amdgcn_mfma_f32_16x16x32_bf16(wbuf[B][q][u], xv, acc[mt][q], 0, 0, 0);   \
        }                                                                                        \
      }                                                                                          \
    }                                                                                            \
  }
  // One stage: stage st+1's x (global -> registers) and the w loads of stage
  // st+DEPTH go out, stage st is multiplied, stage st+1's x goes to the other
  // LDS buffer.  w stage s lives in register buffer s % (DEPTH + 1).
#define NJ_STAGE(B, BN)                                       \
  {                                                           \
    const bool more = st + 1 < st1;                           \
    if (more) NJ_GLOAD_X(st + 1);                             \
    if (st + DEPTH < st1) NJ_LOAD_W(BN, st + DEPTH);          \
    NJ_COMPUTE(B, (st - st0) & 1, st);                        \
    if (more) NJ_SSTORE_X((st + 1 - st0) & 1);                \
    __syncthreads();                                          \
    ++st;                                                     \
    if (st >= st1) break;                                     \
  }

  if constexpr (FULL) {
    // branch-free stage loop (ping-pong over two w register buffers and two x LDS buffers)
#define NJ_FGLOAD_X(st)                                                                          \
  _Pragma("unroll") for (int c = 0; c < PER_T; ++c) {                                            \
    const int idx = threadIdx.x + c * NTH;                                                       \
    const int row = idx / (kStageK / 8), kk = (st) * kStageK + (idx % (kStageK / 8)) * 8;        \
    xr[c] = *reinterpret_cast<const u32x4*>(a.X + (size_t)min(m0 + row, M - 1) * K + kk);        \
  }
#define NJ_FSSTORE_X(buf)                                                                        \
  _Pragma("unroll") for (int c = 0; c < PER_T; ++c) {                                            \
    const int idx = threadIdx.x + c * NTH;                                                       \
    const int row = idx / (kStageK / 8), col = (idx % (kStageK / 8)) * 8;                        \
    *reinterpret_cast<u32x4*>(&xs[buf][row * kRowStride + col]) = xr[c];                         \
  }
#define NJ_FLOAD_W(B, st)                                                                        \
  _Pragma("unroll") for (int u = 0; u < kU; ++u)                                                 \
    _Pragma("unroll") for (int q = 0; q < NG; ++q) wbuf[B][q][u] = ld8(wp[q] + ((st) * kU + u) * 32);
#define NJ_FCOMPUTE(B, buf)                                                                      \
  _Pragma("unroll") for (int u = 0; u < kU; ++u) {                                               \
    _Pragma("unroll") for (int mt = 0; mt < MT; ++mt) {                                          \
      const bf16x8 xv = __builtin_bit_cast(                                                      \
          bf16x8, *reinterpret_cast<const u32x4*>(&xs[buf][(mt * 16 + r) * kRowStride + u * 32 + g * 8])); \
      _Pragma("unroll") for (int q = 0; q < NG; ++q) acc[mt][q] =                                \
          __builtin_amdgcn_mfma_f32_16x16x32_bf16(wbuf[B][q][u], xv, acc[mt][q], 0, 0, 0);       \
    }                                                                                            \
  }
    static_assert(CHUNKS % NTH == 0, "x stage must split evenly over the workgroup");
    NJ_FGLOAD_X(st0);
    NJ_FLOAD_W(0, st0);
    NJ_FSSTORE_X(0);
    __syncthreads();
    for (int st = st0; st < st1; st += 2) {
      const int s1 = min(st + 1, st1 - 1);
      NJ_FGLOAD_X(s1);
      NJ_FLOAD_W(1, s1);
      __builtin_amdgcn_sched_barrier(0);  // keep the loads ahead of the multiplies
      NJ_FCOMPUTE(0, 0);
      NJ_FSSTORE_X(1);
      __syncthreads();
      if (st + 1 >= st1) break;
      const int s2 = min(st + 2, st1 - 1);
      NJ_FGLOAD_X(s2);
      NJ_FLOAD_W(0, s2);
      __builtin_amdgcn_sched_barrier(0);
      NJ_FCOMPUTE(1, 1);
      NJ_FSSTORE_X(0);
      __syncthreads();
    }
#undef NJ_FGLOAD_X
#undef NJ_FSSTORE_X
#undef NJ_FLOAD_W
#undef NJ_FCOMPUTE
  } else if (st0 < st1) {
    NJ_GLOAD_X(st0);
    NJ_LOAD_W(0, st0);
    if (DEPTH > 1 && st0 + 1 < st1) NJ_LOAD_W(1 % (DEPTH + 1), st0 + 1);
    NJ_SSTORE_X(0);
    __syncthreads();
    int st = st0;
    if constexpr (DEPTH == 1) {
      for (;;) {
        NJ_STAGE(0, 1)
        NJ_STAGE(1, 0)
      }
    } else {
      for (;;) {
        NJ_STAGE(0, 2 % (DEPTH + 1))
        NJ_STAGE(1, 3 % (DEPTH + 1))
        NJ_STAGE(2 % (DEPTH + 1), 4 % (DEPTH + 1))
      }
    }
  }
#undef NJ_GLOAD_X
#undef NJ_SSTORE_X
#undef NJ_LOAD_W
#undef NJ_COMPUTE
#undef NJ_STAGE

  const int n = n0 + 4 * g;
  if (nkc > 1) {
    // Split K: publish this chunk's partial, and the last chunk to arrive
    // finishes the tile.  Partials are written and read with device-coherent
    // accesses, so the hand-off needs neither an L2 writeback nor an L2
    // invalidate: each thread waits until its partial stores are acknowledged,
    // then one counter increment publishes them.
    const __amdgpu_buffer_rsrc_t prs = coherent_rsrc(a.part, a.part_bytes);
    auto poff = [&](int j, int m, int q) { return (uint32_t)((((size_t)j * M + m) * NG + q) * Nout + n) * 4u; };
    if (active) {
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const int m = m0 + mt * 16 + r;
        if (m < M)
#pragma unroll
          for (int q = 0; q < NG; ++q) coherent_store(prs, poff(kc, m, q), acc[mt][q]);
      }
    }
    __asm__ volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    int* cnt = a.counters + (size_t)mb * gridDim.x + tile;
    if (threadIdx.x == 0)
      s_last = (__hip_atomic_fetch_add(cnt, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == nkc - 1);
    __syncthreads();
    if (!s_last) return;
    if (threadIdx.x == 0) __hip_atomic_store(cnt, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);  // next launch
    if (!active) return;
    // sum all nkc partials (this workgroup's own included, read back) in chunk order
    for (int j = 0; j < nkc; ++j) {
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const int m = min(m0 + mt * 16 + r, M - 1);  // rows past M: read in range, dropped below
#pragma unroll
        for (int q = 0; q < NG; ++q) {
          const f32x4 v = coherent_load(prs, poff(j, m, q));
          acc[mt][q] = j == 0 ? v : acc[mt][q] + v;
        }
      }
    }
  } else if (!active) {
    return;
  }

#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    const int m = m0 + mt * 16 + r;
    if (m >= M) continue;
    if constexpr (EPI == kEpiStore) {
      *reinterpret_cast<f32x4*>(static_cast<float*>(a.Y) + (size_t)m * Nout + n) = acc[mt][0];
    } else if constexpr (EPI == kEpiResidual) {
      f32x4* p = reinterpret_cast<f32x4*>(static_cast<float*>(a.Y) + (size_t)m * Nout + n);
      *p = *p + acc[mt][0];
    } else {
      const f32x4 gt = acc[mt][0], up = acc[mt][1];
      u32x2 o;
      o[0] = pack_bf16x2(silu_mul(gt[0], up[0]), silu_mul(gt[1], up[1]));
      o[1] = pack_bf16x2(silu_mul(gt[2], up[2]), silu_mul(gt[3], up[3]));
      *reinterpret_cast<u32x2*>(static_cast<bf16_t*>(a.Y) + (size_t)m * Nout + n) = o;
    }
  }
}

// fp32 path (the tiny fp32 model): one wave per output column, lanes split K.
template <int EPI>
__global__ __launch_bounds__(256) void gemm_f32_kernel(const float* __restrict__ X, const float* __restrict__ W,
                                                       void* __restrict__ Y, int M, int Nout, int K) {
  const int lane = threadIdx.x & 63;
  const int n = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (n >= Nout) return;
  const float* w0 = W + (size_t)n * K;
  const float* w1 = W + (size_t)(EPI == kEpiSwiglu ? Nout + n : n) * K;
  for (int m = 0; m < M; ++m) {
    const float* x = X + (size_t)m * K;
    float a0 = 0.f, a1 = 0.f;
    for (int kk = lane; kk < K; kk += 64) {
      a0 = fmaf(x[kk], w0[kk], a0);
      if (EPI == kEpiSwiglu) a1 = fmaf(x[kk], w1[kk], a1);
    }
    for (int o = 32; o > 0; o >>= 1) {
      a0 += __shfl_xor(a0, o);
      if (EPI == kEpiSwiglu) a1 += __shfl_xor(a1, o);
    }
    if (lane == 0) {
      float* y = static_cast<float*>(Y) + (size_t)m * Nout + n;
      if (EPI == kEpiStore) *y = a0;
      else if (EPI == kEpiResidual) *y += a0;
      else *y = silu_mul(a0, a1);
    }
  }
}

template <int MT, int NG, int NW, int EPI>
hipError_t launch_cfg(const GemmK& a, const GemmPlan& p, hipStream_t s) {
  const dim3 grid(p.ntiles, p.mblocks, p.nkc), block(NW * 64);
  const bool full = a.K % kStageK == 0 && (a.Nout / 16) % NW == 0 && a.Nout % 16 == 0;
  if (full)
    hipLaunchKernelGGL((gemm_bf16_kernel<MT, NG, NW, EPI, 1, true>), grid, block, 0, s, a);
  else if (NG == 1 && p.depth == 2)
    hipLaunchKernelGGL((gemm_bf16_kernel<MT, NG, NW, EPI, 2, false>), grid, block, 0, s, a);
  else
    hipLaunchKernelGGL((gemm_bf16_kernel<MT, NG, NW, EPI, 1, false>), grid, block, 0, s, a);
  return hipGetLastError();
}

template <int NG, int EPI>
hipError_t launch_epi(const GemmK& a, const GemmPlan& p, hipStream_t s) {
  if (p.nw == 4) {
    switch (p.mt) {
      case 1: return launch_cfg<1, NG, 4, EPI>(a, p, s);
      case 2: return launch_cfg<2, NG, 4, EPI>(a, p, s);
      case 3: return launch_cfg<3, NG, 4, EPI>(a, p, s);
      default: return launch_cfg<4, NG, 4, EPI>(a, p, s);
    }
  }
  switch (p.mt) {
    case 1: return launch_cfg<1, NG, 8, EPI>(a, p, s);
    case 2: return launch_cfg<2, NG, 8, EPI>(a, p, s);
    case 3: return launch_cfg<3, NG, 8, EPI>(a, p, s);
    default: return launch_cfg<4, NG, 8, EPI>(a, p, s);
  }
}

}  // namespace

static size_t al256(size_t x) { return (x + 255) & ~(size_t)255; }

GemmPlan gemm_tile_plan(int M, int N, int K, int epi, int tile, int nkc) {
  GemmPlan p{};
  const int NG = epi == kEpiSwiglu ? 2 : 1;
  const int Nout = N / NG;
  p.tile = tile;
  const int bm = tile_bm(tile), bno = tile_bn(tile) / NG;
  p.mblocks = (M + bm - 1) / bm;
  p.ntiles = (Nout + bno - 1) / bno;
  const int nst = K / 64;
  p.stages_per_chunk = (nst + nkc - 1) / nkc;
  p.nkc = (nst + p.stages_per_chunk - 1) / p.stages_per_chunk;
  p.depth = 1;
  p.part_bytes = p.nkc > 1 ? al256((size_t)p.nkc * M * N * 4) : 0;
  p.counter_bytes = p.nkc > 1 ? al256((size_t)p.ntiles * p.mblocks * 4) : 0;
  return p;
}

namespace {
// Cost models (seconds) used to pick the kernel for windows of 64+ rows,
// with constants fitted to a sweep of the 8B- and 7B-shaped GEMMs at 64..2048
// rows (the chosen plan is within 15% of the best measured one everywhere).
// Tiled kernel: rounds of resident workgroups times one tile's MFMA time at
// the tile shape's sustained fraction of peak, plus, when K is split, the
// last arriver's reduction (one CU reads nkc partial tiles) and the partial
// traffic.
constexpr double kLaunch = 5e-6;
double tile_cost(const GemmPlan& p, int M, int N, int K) {
  const int bm = tile_bm(p.tile), bn = tile_bn(p.tile);
  const double slots = p.tile == kTile128x128 ? 512.0 : 256.0;  // resident workgroups
  const double eff = p.tile == kTile256x256 ? 0.5 : p.tile == kTile128x256 ? 0.38 : 0.25;
  const double rounds = std::ceil((double)p.ntiles * p.mblocks * p.nkc / slots);
  double t = rounds * 2.0 * bm * bn * (64.0 * p.stages_per_chunk) / (2.5e15 / slots * eff);
  if (p.nkc > 1) t += 2.0 * p.nkc * bm * bn * 4 / 1e11 + 2.0 * p.nkc * (double)M * N * 4 / 5e12;
  return t + kLaunch;
}
// Weight-streaming kernel: one pass over the weights per 64-row block, later
// passes partly served from the caches.
double stream_cost(int M, int N, int K) {
  const int mb = (M + 63) / 64;
  return (double)N * K * 2 * (1.0 + 0.7 * (mb - 1)) / 4e12 + kLaunch;
}
}  // namespace

GemmPlan gemm_tile_choose(int M, int N, int K, int epi, int only_tile) {
  GemmPlan best{};
  double bc = 1e30;
  for (int tile : {kTile256x256, kTile128x256, kTile128x128}) {
    if (only_tile != kTileNone && tile != only_tile) continue;
    for (int nkc = 1; nkc <= 8; nkc *= 2) {
      if (nkc > 1 && K / 64 / nkc < 8) break;
      const GemmPlan p = gemm_tile_plan(M, N, K, epi, tile, nkc);
      if (p.nkc > 1 && (p.counter_bytes > kGemmCounterBytes || p.part_bytes >= kMaxPartBytes)) continue;
      const double c = tile_cost(p, M, N, K);
      if (c < bc) bc = c, best = p;
    }
  }
  return best;
}

bool tile_fits(int M, int N, int K) {
  return K % 64 == 0 && (long)M * K < (1L << 31) && (long)N * K < (1L << 31);
}

GemmPlan gemm_plan(int M, int N, int K, int epi) {
  if (M >= kTileMinRows && tile_fits(M, N, K)) {
    const GemmPlan t = gemm_tile_choose(M, N, K, epi, kTileNone);
    if (tile_cost(t, M, N, K) < stream_cost(M, N, K)) return t;
  }
  return gemm_stream_plan(M, N, K, epi, 0);
}

GemmPlan gemm_stream_plan(int M, int N, int K, int epi, int split) {
  GemmPlan p{};
  p.tile = kTileNone;
  const int NG = epi == kEpiSwiglu ? 2 : 1;
  const int Nout = N / NG;
  p.mt = M >= 64 ? 4 : (M + 15) / 16;
  p.mblocks = (M + p.mt * 16 - 1) / (p.mt * 16);
  const int tiles16 = (Nout + 15) / 16;
  // 8 waves share each staged x tile when it is large and N is wide enough to
  // keep 512+ workgroups; otherwise 4 waves (more workgroups)
  p.nw = (p.mt >= 3 && tiles16 / 8 * p.mblocks >= 512) ? 8 : 4;
  p.ntiles = (tiles16 + p.nw - 1) / p.nw;
  const int nst = (K / 32 + kU - 1) / kU;
  const long base = (long)p.ntiles * p.mblocks;
  // Split K until ~256 workgroups run (one per CU), keeping >= 4 stages per
  // chunk so that the x staging and the partial hand-off are amortised (a
  // measured sweep over the verify step's shapes puts the optimum there).
  int nkc = 1;
  if (split > 0) nkc = std::min(split, nst);
  else
    while (base * nkc * 2 <= kSplitTargetWorkgroups && nst / (nkc * 2) >= 4) nkc *= 2;
  if (split <= 0 && (size_t)nkc * M * N * 4 >= kMaxPartBytes) nkc = 1;
  p.stages_per_chunk = (nst + nkc - 1) / nkc;
  p.nkc = (nst + p.stages_per_chunk - 1) / p.stages_per_chunk;
  p.depth = 1;
  p.part_bytes = p.nkc > 1 ? al256((size_t)p.nkc * M * N * 4) : 0;
  p.counter_bytes = p.nkc > 1 ? al256((size_t)p.ntiles * p.mblocks * 4) : 0;
  static_assert(kSplitTargetWorkgroups / 2 * 4 <= kGemmCounterBytes, "counter region too small");
  return p;
}

hipError_t launch_gemm_plan(const void* x, const void* w, void* y, int M, int N, int K, int epi, const GemmPlan& p,
                            int* counters, float* part, hipStream_t s) {
  if (p.tile != kTileNone) return launch_gemm_tile(x, w, y, M, N, K, epi, p, counters, part, s);
  const int Nout = (epi == kEpiSwiglu) ? N / 2 : N;
  GemmK a{static_cast<const bf16_t*>(x), static_cast<const bf16_t*>(w), y, p.nkc > 1 ? part : nullptr,
          p.nkc > 1 ? counters : nullptr, M, Nout, K, p.stages_per_chunk, (int)p.part_bytes};
  if (epi == kEpiStore) return launch_epi<1, kEpiStore>(a, p, s);
  if (epi == kEpiResidual) return launch_epi<1, kEpiResidual>(a, p, s);
  return launch_epi<2, kEpiSwiglu>(a, p, s);
}

hipError_t launch_gemm(int dtype, const void* x, const void* w, void* y, int M, int N, int K, int epi,
                       int* counters, float* part, hipStream_t s) {
  const int Nout = (epi == kEpiSwiglu) ? N / 2 : N;
  if (dtype == kF32) {
    dim3 grid((Nout + 3) / 4);
    const float* xf = static_cast<const float*>(x);
    const float* wf = static_cast<const float*>(w);
    if (epi == kEpiStore) hipLaunchKernelGGL(gemm_f32_kernel<kEpiStore>, grid, dim3(256), 0, s, xf, wf, y, M, Nout, K);
    else if (epi == kEpiResidual) hipLaunchKernelGGL(gemm_f32_kernel<kEpiResidual>, grid, dim3(256), 0, s, xf, wf, y, M, Nout, K);
    else hipLaunchKernelGGL(gemm_f32_kernel<kEpiSwiglu>, grid, dim3(256), 0, s, xf, wf, y, M, Nout, K);
    return hipGetLastError();
  }
  return launch_gemm_plan(x, w, y, M, N, K, epi, gemm_plan(M, N, K, epi), counters, part, s);
}

}  // namespace nj
