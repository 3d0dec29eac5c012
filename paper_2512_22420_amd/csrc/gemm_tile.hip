// Large-window GEMMs (M = B*(k+1) in the hundreds or thousands): y = x . w^T
// with both operands staged through LDS.
//
// Above M ~ 300 rows the verify step's GEMMs are bound by the matrix cores
// (2*M FLOP per weight byte against a 312 FLOP/byte ridge), so the
// weight-streaming kernel, which re-reads the weights once per 64 window rows
// and feeds every MFMA with one LDS read, is the wrong shape.  Here a
// workgroup owns a BM x BN output tile (x rows x weight rows), stages 64-wide
// K slices of both operands in LDS (double-buffered, 16-byte row pad), and
// each wave multiplies a (BM/WM) x (BN/WN) sub-tile with 16x16x32 bf16 MFMAs,
// so every LDS fragment read feeds TN (or TM) MFMAs.
//
// - Tile order is XCD-aware: workgroup IDs go round-robin over the 8 XCDs, so
//   the linear ID is remapped to give each XCD a contiguous run of tiles, with
//   the M tiles of one weight tile adjacent.  The weight tile is then fetched
//   from HBM once and re-read by its neighbours from that XCD's L2.
// - When there are too few tiles to fill the chip, K is split across
//   workgroups with the same fixed-order, last-arriver reduction as the
//   weight-streaming kernel.
// - Epilogues as in the weight-streaming kernel: fp32 store, fp32 residual
//   add, and SwiGLU, for which the first half of the weight tile holds gate
//   rows and the second half the matching up rows.
#include "common.h"
#include "kernels.h"

namespace nj {
namespace {


__device__ __forceinline__ float silu_mul(float gte, float up) { return gte / (1.0f + expf(-gte)) * up; }

struct TileK {
  const bf16_t* X;
  const bf16_t* W;
  void* Y;
  float* part;    // [nkc][M][NG][Nout] fp32 partials (split K only)
  int* counters;  // [tiles_n * tiles_m][kCounterStride] arrival counters (split K only), zero between launches
  int M, Nout, K, tiles_m, tiles_n, nkc, stages_per_chunk;
  int part_bytes;
};

// BK: K per stage (32 or 64); LDS rows are padded by 16 bytes, which keeps
// the 16-byte fragment reads of 8 consecutive rows on distinct banks.  DIST:
// stages loaded ahead of the one being multiplied (1 or 2).
template <int BM, int BN, int WM, int WN, int BK, int DIST, int LAYOUT, int PIPE, int NG, int EPI>
__global__ __launch_bounds__(WM * WN * 64) void gemm_tile_kernel(TileK a) {
  constexpr int kBK = BK;
  constexpr int PR = BK / 8;                       // 16-byte pieces per row and stage
  constexpr int kLdsStride = LAYOUT == 0 ? BK + 8 : BK;
  constexpr int NTH = WM * WN * 64;
  constexpr int TM = BM / WM / 16;                 // x fragments per wave
  constexpr int TN = BN / WN / 16;                 // weight fragments per wave
  constexpr int XC = BM * PR / NTH;                // 16-byte x pieces per thread per stage
  constexpr int WC = BN * PR / NTH;
  constexpr int HALF = BN / 2;                     // SwiGLU: gate rows, then up rows
  static_assert(XC * NTH == BM * PR && WC * NTH == BN * PR, "stage must split evenly");
  static_assert(NG == 1 || (TN % 2 == 0), "SwiGLU waves hold gate and up fragments in pairs");
  // LDS element offset of 16-byte piece `ch` of tile row `row`
  auto lds_off = [](int row, int ch) {
    if constexpr (LAYOUT == 0) return row * kLdsStride + ch * 8;
    else if constexpr (LAYOUT == 1) {
      const int f = PR == 8 ? ((row >> 1) ^ ((row & 1) << 2)) : ((row >> 1) ^ (row >> 3));
      return row * kLdsStride + ((ch ^ f) & (PR - 1)) * 8;
    } else {
      return row * kLdsStride + ((ch ^ row) & (PR - 1)) * 8;
    }
  };
  __shared__ __attribute__((aligned(16))) bf16_t xs[2][BM * kLdsStride];
  __shared__ __attribute__((aligned(16))) bf16_t ws[2][BN * kLdsStride];
  __shared__ int s_last;

  // XCD-aware tile order: workgroup b runs on XCD b % 8; XCD x takes the
  // x-th contiguous share of the logical tiles.
  const int total = a.tiles_m * a.tiles_n * a.nkc;
  const int bid = blockIdx.x;
  const int per = total >> 3, rem = total & 7, xcd = bid & 7, loc = bid >> 3;
  const int t = xcd < rem ? xcd * (per + 1) + loc : rem * (per + 1) + (xcd - rem) * per + loc;
  const int tm = t % a.tiles_m;
  const int tk = t / a.tiles_m;
  const int kc = tk % a.nkc;
  const int tn = tk / a.nkc;

  const int M = a.M, Nout = a.Nout, K = a.K;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int r = lane & 15, g = lane >> 4;
  const int m0 = tm * BM;
  const int n0 = tn * (NG == 1 ? BN : HALF);

  // element offsets of this thread's 16-byte pieces (row clamped into range;
  // rows past the end are computed and never stored).  Both operands hold
  // fewer than 2^31 elements (checked by the host).
  uint32_t xo[XC], wo[WC];
#pragma unroll
  for (int c = 0; c < XC; ++c) {
    const int idx = threadIdx.x + c * NTH, row = idx / PR;
    xo[c] = (uint32_t)min(m0 + row, M - 1) * (uint32_t)K + (idx % PR) * 8;
  }
  // Weight pieces come from the packed layout (128-row groups, k-step major,
  // 1 KB per 16-row x 32-k tile in MFMA lane order): thread piece idx is lane
  // idx % 64 of k-step (idx / 64) % KSS of 16-row tile idx / (64 * KSS), so
  // each wave reads whole 1 KB tiles.  Tiles past the edge are clamped to the
  // last one (computed and never stored).
  constexpr int KSS = kBK / 32;  // k-steps per stage
  const int KS = K / 32, nto = Nout / 16;
#pragma unroll
  for (int c = 0; c < WC; ++c) {
    const int idx = threadIdx.x + c * NTH;
    const int t16 = idx / (64 * KSS), ksl = (idx / 64) % KSS, ln = idx % 64;
    int T;
    if constexpr (NG == 1) T = min(n0 / 16 + t16, nto - 1);
    else T = t16 < HALF / 16 ? min(n0 / 16 + t16, nto - 1) : nto + min(n0 / 16 + t16 - HALF / 16, nto - 1);
    wo[c] = ((uint32_t)(T >> 3) * (uint32_t)KS * 8u + (uint32_t)(T & 7)) * 512u + (uint32_t)ksl * 4096u + ln * 8;
  }
  auto w_lds = [&](int idx) {  // LDS element offset of weight piece idx
    const int t16 = idx / (64 * KSS), ksl = (idx / 64) % KSS, ln = idx % 64;
    return lds_off(t16 * 16 + (ln & 15), ksl * 4 + (ln >> 4));
  };

  // LDS row of weight fragment j of this wave
  auto wrow = [&](int j) {
    if constexpr (NG == 1) return wn * (BN / WN) + j * 16;
    else return (j < TN / 2) ? wn * (HALF / WN) + j * 16 : HALF + wn * (HALF / WN) + (j - TN / 2) * 16;
  };

  f32x4 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  // the plan counts K in 64-wide stages
  const int nst = K / kBK, spc = a.stages_per_chunk * (64 / kBK);
  const int st0 = kc * spc, st1 = min(nst, st0 + spc);

  // DIST register sets: with two, the loads of stage s+2 are in flight while
  // stage s is multiplied and stage s+1 is copied into LDS.
  u32x4 xr[DIST][XC], wr[DIST][WC];
  auto gload = [&](int set, int st) {
    const int k0 = st * kBK;
#pragma unroll
    for (int c = 0; c < XC; ++c) xr[set][c] = *reinterpret_cast<const u32x4*>(a.X + (xo[c] + k0));
#pragma unroll
    for (int c = 0; c < WC; ++c) wr[set][c] = *reinterpret_cast<const u32x4*>(a.W + (wo[c] + (uint32_t)st * (KSS * 4096u)));
  };
  auto sstore = [&](int set, int buf) {
#pragma unroll
    for (int c = 0; c < XC; ++c) {
      const int idx = threadIdx.x + c * NTH;
      *reinterpret_cast<u32x4*>(&xs[buf][lds_off(idx / PR, idx % PR)]) = xr[set][c];
    }
#pragma unroll
    for (int c = 0; c < WC; ++c) *reinterpret_cast<u32x4*>(&ws[buf][w_lds(threadIdx.x + c * NTH)]) = wr[set][c];
  };
  auto compute = [&](int buf) {
    constexpr int KS = kBK / 32;
    if constexpr (PIPE == 2) {
      // per k-step: TN+2 reads ahead, then two more reads per group of TN multiplies
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        bf16x8 xf[TM], wf[TN];
#pragma unroll
        for (int j = 0; j < TN; ++j)
          wf[j] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(
                                                 &ws[buf][lds_off(wrow(j) + r, ks * 4 + g)]));
#pragma unroll
        for (int i = 0; i < TM; ++i)
          xf[i] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(
                                                 &xs[buf][lds_off(wm * (BM / WM) + i * 16 + r, ks * 4 + g)]));
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf[j], xf[i], acc[i][j], 0, 0, 0);
        constexpr int REM = TM - 2, N2 = REM / 2;
        __builtin_amdgcn_sched_group_barrier(0x100, TN + 2, 0);
#pragma unroll
        for (int q = 0; q < N2; ++q) {
          __builtin_amdgcn_sched_group_barrier(0x008, TN, 0);
          __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
        }
        if constexpr (REM & 1) {
          __builtin_amdgcn_sched_group_barrier(0x008, TN, 0);
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        }
#pragma unroll
        for (int q = N2 + (REM & 1); q < TM; ++q) __builtin_amdgcn_sched_group_barrier(0x008, TN, 0);
      }
    } else if constexpr (PIPE == 0) {
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        bf16x8 xf[TM], wf[TN];
#pragma unroll
        for (int i = 0; i < TM; ++i)
          xf[i] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(
                                                 &xs[buf][lds_off(wm * (BM / WM) + i * 16 + r, ks * 4 + g)]));
#pragma unroll
        for (int j = 0; j < TN; ++j)
          wf[j] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(
                                                 &ws[buf][lds_off(wrow(j) + r, ks * 4 + g)]));
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf[j], xf[i], acc[i][j], 0, 0, 0);
      }
    } else {
      // Fragment reads run ahead of the multiplies: the stage's reads are
      // issued in use order (per k-step: weight fragments, then x fragments),
      // and the scheduler is held to "TN+2 reads, then per group of TN
      // multiplies two more reads", so each LDS read has at least one MFMA
      // group (and the other wave on the SIMD) to hide its latency.
      bf16x8 xf[KS][TM], wf[KS][TN];
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
#pragma unroll
        for (int j = 0; j < TN; ++j)
          wf[ks][j] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(
                                                     &ws[buf][lds_off(wrow(j) + r, ks * 4 + g)]));
#pragma unroll
        for (int i = 0; i < TM; ++i)
          xf[ks][i] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(
                                                     &xs[buf][lds_off(wm * (BM / WM) + i * 16 + r, ks * 4 + g)]));
      }
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf[ks][j], xf[ks][i], acc[i][j], 0, 0, 0);
      constexpr int R = KS * (TM + TN), INIT = TN + 2, REM = R - INIT, G = KS * TM, N2 = REM / 2;
      static_assert(N2 + (REM & 1) <= G, "read schedule longer than the multiplies");
      __builtin_amdgcn_sched_group_barrier(0x100, INIT, 0);
#pragma unroll
      for (int q = 0; q < N2; ++q) {
        __builtin_amdgcn_sched_group_barrier(0x008, TN, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
      }
      if constexpr (REM & 1) {
        __builtin_amdgcn_sched_group_barrier(0x008, TN, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      }
#pragma unroll
      for (int q = N2 + (REM & 1); q < G; ++q) __builtin_amdgcn_sched_group_barrier(0x008, TN, 0);
    }
  };

  // Branch-free double-buffered stage loops (the last iterations re-load the
  // last stage into buffers nobody reads, an L2 hit; branches inside the loop
  // would make the compiler drain the loads in flight at every join).
  if constexpr (DIST == 1) {
    gload(0, st0);
    sstore(0, 0);
    __syncthreads();
    for (int st = st0; st < st1; ++st) {
      const int buf = (st - st0) & 1;
      gload(0, min(st + 1, st1 - 1));
      __builtin_amdgcn_sched_barrier(0);
      compute(buf);
      sstore(0, buf ^ 1);
      __syncthreads();
    }
  } else {
    // register set q and LDS buffer q alternate; stage st + 2 is loaded while
    // stage st is multiplied and stage st + 1 goes from registers to LDS
    gload(0, st0);
    gload(1, min(st0 + 1, st1 - 1));
    sstore(0, 0);
    __syncthreads();
    for (int st = st0; st < st1; st += 2) {
      gload(0, min(st + 2, st1 - 1));
      __builtin_amdgcn_sched_barrier(0);
      compute(0);
      sstore(1, 1);
      __syncthreads();
      if (st + 1 >= st1) break;
      gload(1, min(st + 3, st1 - 1));
      __builtin_amdgcn_sched_barrier(0);
      compute(1);
      sstore(0, 0);
      __syncthreads();
    }
  }

  // output coordinates of fragment (i, j): row m(i), columns n(j)..n(j)+3 of group q(j)
  auto out_m = [&](int i) { return m0 + wm * (BM / WM) + i * 16 + r; };
  auto out_n = [&](int j) {
    if constexpr (NG == 1) return n0 + wn * (BN / WN) + j * 16 + 4 * g;
    else return n0 + wn * (HALF / WN) + (j % (TN / 2)) * 16 + 4 * g;
  };
  auto out_q = [&](int j) { return NG == 1 ? 0 : j / (TN / 2); };

  if (a.nkc > 1) {
    // Split K: publish the partial with device-coherent stores, count arrivals,
    // and let the last workgroup of the tile add the partials in chunk order.
    const __amdgpu_buffer_rsrc_t prs = coherent_rsrc(a.part, a.part_bytes);
    auto poff = [&](int c, int m, int j) {
      return (uint32_t)((((size_t)c * M + m) * NG + out_q(j)) * Nout + out_n(j)) * 4u;
    };
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const int m = out_m(i);
      if (m >= M) continue;
#pragma unroll
      for (int j = 0; j < TN; ++j)
        if (out_n(j) < Nout) coherent_store(prs, poff(kc, m, j), acc[i][j]);
    }
    __asm__ volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    int* cnt = a.counters + ((size_t)tn * a.tiles_m + tm) * kCounterStride;
    if (threadIdx.x == 0)
      s_last = (__hip_atomic_fetch_add(cnt, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == a.nkc - 1);
    __syncthreads();
    if (!s_last) return;
    if (threadIdx.x == 0) __hip_atomic_store(cnt, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);  // next launch
    // Sum all nkc partials (this workgroup's own included, read back) in chunk
    // order; half of the fragments at a time keeps 16 loads in flight.
    // Fragments past the edge read a clamped in-range address and are dropped.
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      for (int c = 0; c < a.nkc; ++c) {
#pragma unroll
        for (int i = h * (TM / 2); i < (h + 1) * (TM / 2); ++i) {
          const int m = min(out_m(i), M - 1);
#pragma unroll
          for (int j = 0; j < TN; ++j) {
            const uint32_t off = (uint32_t)((((size_t)c * M + m) * NG + out_q(j)) * Nout + min(out_n(j), Nout - 4)) * 4u;
            const f32x4 v = coherent_load(prs, off);
            acc[i][j] = c == 0 ? v : acc[i][j] + v;
          }
        }
      }
    }
  }

#pragma unroll
  for (int i = 0; i < TM; ++i) {
    const int m = out_m(i);
    if (m >= M) continue;
#pragma unroll
    for (int j = 0; j < (NG == 1 ? TN : TN / 2); ++j) {
      const int n = out_n(j);
      if (n >= Nout) continue;
      if constexpr (EPI == kEpiStore) {
        *reinterpret_cast<f32x4*>(static_cast<float*>(a.Y) + (size_t)m * Nout + n) = acc[i][j];
      } else if constexpr (EPI == kEpiResidual) {
        f32x4* p = reinterpret_cast<f32x4*>(static_cast<float*>(a.Y) + (size_t)m * Nout + n);
        *p = *p + acc[i][j];
      } else {
        const f32x4 gt = acc[i][j], up = acc[i][j + TN / 2];
        u32x2 o;
        o[0] = pack_bf16x2(silu_mul(gt[0], up[0]), silu_mul(gt[1], up[1]));
        o[1] = pack_bf16x2(silu_mul(gt[2], up[2]), silu_mul(gt[3], up[3]));
        *reinterpret_cast<u32x2*>(static_cast<bf16_t*>(a.Y) + (size_t)m * Nout + n) = o;
      }
    }
  }
}

template <int BM, int BN, int WM, int WN, int BK, int DIST, int LAYOUT, int PIPE>
hipError_t launch_shape(const TileK& a, int epi, hipStream_t s) {
  const dim3 grid(a.tiles_m * a.tiles_n * a.nkc), block(WM * WN * 64);
  if (epi == kEpiStore) hipLaunchKernelGGL((gemm_tile_kernel<BM, BN, WM, WN, BK, DIST, LAYOUT, PIPE, 1, kEpiStore>), grid, block, 0, s, a);
  else if (epi == kEpiResidual)
    hipLaunchKernelGGL((gemm_tile_kernel<BM, BN, WM, WN, BK, DIST, LAYOUT, PIPE, 1, kEpiResidual>), grid, block, 0, s, a);
  else hipLaunchKernelGGL((gemm_tile_kernel<BM, BN, WM, WN, BK, DIST, LAYOUT, PIPE, 2, kEpiSwiglu>), grid, block, 0, s, a);
  return hipGetLastError();
}

}  // namespace

int tile_bm(int cfg) { return cfg == kTile256x256 ? 256 : 128; }
int tile_bn(int cfg) { return cfg == kTile128x128 ? 128 : 256; }

hipError_t launch_gemm_tile(const void* x, const void* w, void* y, int M, int N, int K, int epi, const GemmPlan& p,
                            int* counters, float* part, hipStream_t s) {
  const int Nout = (epi == kEpiSwiglu) ? N / 2 : N;
  TileK a{static_cast<const bf16_t*>(x), static_cast<const bf16_t*>(w), y, p.nkc > 1 ? part : nullptr,
          p.nkc > 1 ? counters : nullptr, M, Nout, K, p.mblocks, p.ntiles, p.nkc, p.stages_per_chunk,
          (int)p.part_bytes};
  switch (p.tile) {
    case kTile256x256: return launch_shape<256, 256, 2, 4, 64, 2, 1, 2>(a, epi, s);
    case kTile128x256: return launch_shape<128, 256, 2, 4, 64, 2, 1, 1>(a, epi, s);
    default: return launch_shape<128, 128, 2, 2, 64, 1, 1, 0>(a, epi, s);
  }
}

}  // namespace nj
