// GEMMs of the verify step: y = x . w^T over the B*(k+1) window rows.
//
// bf16 path: weight-streaming MFMA kernel.  At verify-step sizes M = B*(k+1)
// is 1..~768 while N*K reaches 5e8 (LM head), so below M ~ 300 the work is
// bound by reading each weight byte once from HBM.
//
// Weights are read in the packed layout of pack_weight_kernel (below): 128-row
// groups, each one contiguous run of K/32 k-steps, each k-step 8 row tiles of
// 16 rows x 32 k, and each tile exactly the 1 KB that the 64 lanes of a wave
// load as the A operand of v_mfma_f32_16x16x32_bf16 (lane l: row l & 15,
// k (l >> 4) * 8 .. +8).  So every weight load instruction reads 1 KB
// contiguous, the 8 waves of a workgroup read 8 KB contiguous per k-step, and
// each workgroup streams one contiguous region -- the access pattern that
// gets closest to the HBM read ceiling on this part (a row-major matrix read
// in 16-row tiles leaves ~10% of the bandwidth unused).
//
// - Weights are read once per step, so their loads are non-temporal (streaming
//   loads that do not displace cached data; measured 8-12% faster on the
//   LM-head stream than plain loads).
// - Each wave owns one 16-row weight tile (gate and up tiles are two waves of
//   one workgroup for SwiGLU) and streams it along K in stages of 4 k-steps,
//   with the next stage's loads in flight while the current one is
//   multiplied (two register sets, a branch-free loop: stages past the end of
//   the K range re-read the last stage and see zero activations).
// - The activation rows (B operand, M padded to 16) are staged per stage in
//   LDS, loaded once per workgroup and shared by its 8 waves.  The x loads of
//   a stage are issued before its weight loads, so the wait that puts x into
//   LDS never waits for weight loads issued after it.
// - When the tiles alone give too few workgroups to fill 256 CUs (small N),
//   K is split across workgroups: each writes an fp32 partial, and the last
//   workgroup of a tile to arrive (device-scope counter) adds the partials in
//   chunk order and applies the epilogue, so results do not depend on arrival
//   order.  Counters reset themselves for the next launch.
// - Epilogues: store fp32, add into the fp32 residual stream, or SwiGLU
//   (the up waves hand their accumulators to the gate waves through LDS),
//   stored as bf16.
//
// Result layout (16x16x32 bf16): lane l holds weight rows 4*(l >> 4) + i,
// x row l & 15.  Any k permutation applied to both operands leaves the
// product unchanged.
#include <algorithm>
#include <cmath>
#include <cstdlib>
#include <mutex>
#include <unordered_map>
#include <utility>

#include "common.h"
#include "kernels.h"

namespace nj {
namespace {

constexpr int kSU = 4;                   // 32-wide k-steps per stage
constexpr int kSK = 32 * kSU;            // 128 k per stage
constexpr int kXStride = kSK + 8;        // LDS row stride in elements (+16 bytes)
constexpr int kNW = 8;                   // waves per workgroup
constexpr int kSplitTargetWorkgroups = 256;
constexpr int kRedBatch = 4;             // split-K partials loaded together by the reducing workgroup

__device__ __forceinline__ float silu_mul(float gte, float up) { return gte / (1.0f + expf(-gte)) * up; }

struct GemmK {
  const bf16_t* X;
  const bf16_t* W;  // packed
  void* Y;
  float* part;      // [nkc][M][N] fp32 partials (split K only; column = weight row)
  int* counters;    // [mblocks][gridDim.x][kCounterStride] arrival counters (split K only), zero between launches
  int M, Nout, K, KS, stages_per_chunk;
  int part_bytes;
  float* stats;     // kEpiLogits: [M][nch][2] chunk max and sum of exp (chunk = this kernel's 128 columns)
  int nch;
  // RMSNorm folded into the GEMMs.  Input side (any epilogue but the
  // residual ones): x holds h * gain, and row m of the product is scaled by
  // 1 / sqrt(sum_t ssq_in[m][t] / K + eps).  Output side (kEpiResidualNorm):
  // besides h += acc, write xg = bf16(h * gain) and ssq_out[m][tile] = sum of
  // h^2 over the workgroup's 128 columns, the next GEMM's input side.
  const float* ssq_in;
  int nt_in;
  float eps;
  const bf16_t* gain;
  bf16_t* xg;
  float* ssq_out;
  QkvRope rope;     // kEpiQkvRope
  int ykbM;         // kEpiSwiglu: nonzero = y stored k-blocked, [Nout/32][M][32] (M = ykbM)
  int par;          // split K: every chunk's workgroup reduces and finishes a slice of the block's rows
  int par_l2;       // par, and round-robin dispatch puts every chunk of a block on one XCD (see below)
  unsigned foreign; // chunks that act as if dispatched elsewhere (tests of the fallback; normally 0)
  int xg_kb;        // kEpiResidualNorm: xg stored k-blocked, [Nout/32][M][32]
};

// The weight stream of one 16-row weight tile (wp: this lane's piece of k-step
// 0) over stages [st0, st1), accumulated into acc.  NB register sets: the
// loads of stages st+1 .. st+NB-1 are in flight while stage st is multiplied.
// The x pieces of a stage go through LDS (two buffers of ROWS x kXStride at
// xs); each thread owns PT of them (xp: row base, xc: column in the stage, xo:
// LDS offset).  Ends on a barrier, so LDS is free afterwards.
template <int MT, int NB, int PT>
__device__ __forceinline__ void stream_tile(f32x4 (&acc)[MT], const bf16_t* wp, const bf16_t* const (&xp)[PT],
                                            const int (&xc)[PT], const int (&xo)[PT], int K, int KS, int st0,
                                            int st1, bf16_t* xs) {
  constexpr int XB = MT * 16 * kXStride;  // one LDS buffer
  const int lane = threadIdx.x & 63, r = lane & 15, g = lane >> 4;
  const int last = st1 - 1;
  u32x4 xr[NB][PT];
  bf16x8 wb[NB][kSU];

  auto loadx = [&](auto setc, int st) {
    constexpr int set = decltype(setc)::value;
#pragma unroll
    for (int c = 0; c < PT; ++c)
      xr[set][c] = *reinterpret_cast<const u32x4*>(xp[c] + min(st * kSK + xc[c], K - 8));
  };
  auto loadw = [&](auto setc, int st) {
    constexpr int set = decltype(setc)::value;
#pragma unroll
    for (int u = 0; u < kSU; ++u)
      wb[set][u] = __builtin_bit_cast(
          bf16x8, __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(wp + (size_t)min(st * kSU + u, KS - 1) * 4096)));
  };
  // x of stage st into LDS buffer buf; zero past the chunk or past K
  auto storex = [&](auto setc, int buf, int st) {
    constexpr int set = decltype(setc)::value;
#pragma unroll
    for (int c = 0; c < PT; ++c) {
      const uint32_t keep = 0u - (uint32_t)(st < st1 && st * kSK + xc[c] < K);  // all ones or zero
      *reinterpret_cast<u32x4*>(&xs[buf * XB + xo[c]]) = xr[set][c] & keep;
    }
  };
  // The x fragments of k-step u+1 are read from LDS while k-step u is
  // multiplied (two register sets): left to itself the scheduler waits for
  // each LDS read right before its MFMA, which serialises the read latencies.
  auto compute = [&](auto setc, int buf) {
    constexpr int set = decltype(setc)::value;
    bf16x8 xv[2][MT];
    auto rd = [&](int slot, int u) {
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
        xv[slot][mt] = __builtin_bit_cast(
            bf16x8, *reinterpret_cast<const u32x4*>(&xs[buf * XB + (mt * 16 + r) * kXStride + u * 32 + g * 8]));
    };
    rd(0, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, MT, 0);
#pragma unroll
    for (int u = 0; u < kSU; ++u) {
      if (u + 1 < kSU) rd((u + 1) & 1, u + 1);
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
        acc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wb[set][u], xv[u & 1][mt], acc[mt], 0, 0, 0);
      if (u + 1 < kSU) __builtin_amdgcn_sched_group_barrier(0x100, MT, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, MT, 0);
    }
  };
  // prologue: stages st0 .. st0+NB-2 in flight, stage st0's x in LDS buffer 0
  [&]<int... I>(std::integer_sequence<int, I...>) {
    ((loadx(std::integral_constant<int, I>{}, min(st0 + I, last)),
      loadw(std::integral_constant<int, I>{}, min(st0 + I, last))), ...);
  }(std::make_integer_sequence<int, NB - 1>{});
  storex(std::integral_constant<int, 0>{}, 0, st0);
  __syncthreads();
  // stage t = st + J uses register set J and LDS buffer J & 1 (NB is even);
  // it issues the loads of stage t + NB - 1 into set (J + NB - 1) % NB, which
  // stage t - 1 has finished with
  for (int st = st0; st < st1; st += NB) {
    [&]<int... J>(std::integer_sequence<int, J...>) {
      ([&] {
        constexpr int nxt = (J + NB - 1) % NB;
        const int t = st + J;
        // issue order pinned: x before the weights (the in-order load counter
        // then lets the x wait leave the weight loads in flight), both ahead
        // of the multiplies
        __builtin_amdgcn_sched_barrier(0);
        loadx(std::integral_constant<int, nxt>{}, min(t + NB - 1, last));
        __builtin_amdgcn_sched_barrier(0);
        loadw(std::integral_constant<int, nxt>{}, min(t + NB - 1, last));
        __builtin_amdgcn_sched_barrier(0);
        compute(std::integral_constant<int, J>{}, J & 1);
        storex(std::integral_constant<int, (J + 1) % NB>{}, (J + 1) & 1, t + 1);
        __syncthreads();
      }(), ...);
    }(std::make_integer_sequence<int, NB>{});
  }
}

template <int MT, int EPI, int NB>
__global__ __launch_bounds__(kNW * 64) void gemm_stream_kernel(GemmK a) {
  constexpr int NG = EPI == kEpiSwiglu ? 2 : 1;
  constexpr int TPW = kNW / NG;                   // output tiles per workgroup
  static_assert(EPI != kEpiLogits || TPW * 16 == kStatChunk, "a workgroup's columns are one statistics chunk");
  static_assert(EPI != kEpiResidualNorm || TPW * 4 == 32, "a row segment is 32 lanes");
  static_assert(EPI != kEpiQkvRope || TPW * 16 == 128, "a workgroup's columns are one head");
  constexpr int ROWS = MT * 16, NTH = kNW * 64;
  constexpr int CH = ROWS * (kSK / 8);            // 16-byte x pieces per stage
  constexpr int PT = (CH + NTH - 1) / NTH;
  __shared__ __attribute__((aligned(16))) bf16_t xs[2][ROWS * kXStride];
  __shared__ int s_last;

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r = lane & 15, g = lane >> 4;
  const int M = a.M, Nout = a.Nout, K = a.K, KS = a.KS;
  const int mb = blockIdx.y, kc = blockIdx.z, nkc = gridDim.z;
  const int m0 = mb * ROWS;
  const int nto = Nout / 16;                       // output tiles
  const int otile = blockIdx.x * TPW + wave % TPW;
  const bool active = otile < nto;
  const int half = NG == 1 ? 0 : wave / TPW;       // 0: gate (or plain) tile, 1: up tile
  const int wtile = half * nto + min(otile, nto - 1);
  const bf16_t* wp = a.W + ((size_t)(wtile >> 3) * KS * 8 + (wtile & 7)) * 512 + lane * 8;

  const int nst = (KS + kSU - 1) / kSU;
  const int st0 = kc * a.stages_per_chunk, st1 = min(nst, st0 + a.stages_per_chunk);

  // this thread's x pieces: row, 8-element column of the stage
  const bf16_t* xp[PT];
  int xo[PT], xc[PT];
#pragma unroll
  for (int c = 0; c < PT; ++c) {
    const int idx = min((int)threadIdx.x + c * NTH, CH - 1);  // surplus threads repeat the last piece
    const int row = idx / (kSK / 8), col = (idx % (kSK / 8)) * 8;
    xp[c] = a.X + (size_t)min(m0 + row, M - 1) * K;
    xc[c] = col;
    xo[c] = row * kXStride + col;
  }

  // Loads only the epilogue needs are issued first, so that they complete
  // under the weight stream instead of adding a round trip at either end.
  // Input-side norm: this thread's 8 sums-of-squares partials (8 lanes per
  // row; lane c takes partials c, c+8, ...).
  __shared__ float s_rinv[ROWS];
  const bool scaled = a.ssq_in != nullptr;
  float ssq_v[8];
  if (scaled) {
    const int row = min((int)threadIdx.x / 8, ROWS - 1), c = threadIdx.x % 8;
    const float* sp = a.ssq_in + (size_t)min(m0 + row, M - 1) * a.nt_in;
#pragma unroll
    for (int j = 0; j < 8; ++j) ssq_v[j] = c + 8 * j < a.nt_in ? sp[c + 8 * j] : 0.f;
  }
  // QKV + RoPE epilogue: the (cos, sin) of this thread's rotation units
  // (unit u = thread + it * NTH: row u / 64, pair u % 64).
  constexpr int RP_IT = (ROWS * 64 + NTH - 1) / NTH;
  u32x2 cs_pre[EPI == kEpiQkvRope ? RP_IT : 1];
  if constexpr (EPI == kEpiQkvRope) {
#pragma unroll
    for (int it = 0; it < RP_IT; ++it) {
      const int u = threadIdx.x + it * NTH;
      const int m = min(m0 + u / 64, M - 1), j = u % 64;
      cs_pre[it] = *reinterpret_cast<const u32x2*>(a.rope.cs + ((size_t)m * 64 + j) * 2);
    }
  }
  // Residual-norm epilogue: the residual rows and gains of this thread's
  // output pieces (see the epilogue for the piece layout).
  constexpr int RN_PIECES = ROWS * TPW * 4, RN_IT = (RN_PIECES + NTH - 1) / NTH;
  f32x4 h_pre[EPI == kEpiResidualNorm ? RN_IT : 1];
  u32x2 g_pre[EPI == kEpiResidualNorm ? RN_IT : 1];
  if constexpr (EPI == kEpiResidualNorm) {
    const int n0 = blockIdx.x * TPW * 16;
#pragma unroll
    for (int it = 0; it < RN_IT; ++it) {
      const int idx = threadIdx.x + it * NTH;
      const int row = idx / (TPW * 4), c4 = (idx % (TPW * 4)) * 4;
      const int m = min(m0 + row, M - 1), n = min(n0 + c4, Nout - 4);
      h_pre[it] = *reinterpret_cast<const f32x4*>(static_cast<const float*>(a.Y) + (size_t)m * Nout + n);
      g_pre[it] = *reinterpret_cast<const u32x2*>(a.gain + n);
    }
  }

  f32x4 acc[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) acc[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
  stream_tile<MT, NB, PT>(acc, wp, xp, xc, xo, K, KS, st0, st1, &xs[0][0]);

  const int ncol = wtile * 16 + 4 * g;  // weight rows of this lane's results
  // rows [mlo, mhi) of the window are this workgroup's to finish (all of the
  // block's, but for the slice-reduced split K)
  int mlo = m0, mhi = min(M, m0 + ROWS);
  if (nkc > 1) {
    // Split K: publish this chunk's partial, and the last chunk to arrive
    // finishes the tile.  Partials are written and read with device-coherent
    // accesses, so the hand-off needs neither an L2 writeback nor an L2
    // invalidate: each thread waits until its partial stores are acknowledged,
    // then one counter increment publishes them.
    // With par_l2 the host has laid the grid out so that round-robin dispatch
    // (workgroup i to XCD i mod 8) puts every chunk of a block on one XCD;
    // a chunk that finds itself there exchanges its partial through that
    // XCD's L2 (xcd_store / xcd_load), one that does not ("foreign") writes
    // through to memory and says so with its arrival (bit 16 + kc of the
    // counter), so that its partial is read from memory and, when the block's
    // chunks are mixed, one chunk that is on the expected XCD finishes the
    // whole block.  The sums are the same in every case.
    const int Ntot = Nout * NG;
    const __amdgpu_buffer_rsrc_t prs = coherent_rsrc(a.part, a.part_bytes);
    auto poff = [&](int j, int m) { return (uint32_t)(((size_t)j * M + m) * Ntot + ncol) * 4u; };
    const unsigned lbid = blockIdx.x + gridDim.x * (blockIdx.y + gridDim.y * blockIdx.z);
    const bool foreign = a.par_l2 && (xcd_id() != (lbid & 7u) || ((a.foreign >> kc) & 1u));
    const bool l2 = a.par_l2 && !foreign;
    if (active) {
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const int m = m0 + mt * 16 + r;
        if (m < M) {
          if (l2) xcd_store(prs, poff(kc, m), acc[mt]);
          else coherent_store(prs, poff(kc, m), acc[mt]);
        }
      }
    }
    __asm__ volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    int* cnt = a.counters + ((size_t)mb * gridDim.x + blockIdx.x) * kCounterStride;
    if (a.par) {
      // Every chunk's workgroup waits for all nkc partials of the tile, then
      // sums rows [mlo, mhi) of the block over them in chunk order (the same
      // additions as the last-arriver form, so the same bits) and runs the
      // epilogue on those rows only.  The host runs this only when every
      // workgroup of the grid has a CU of its own; the wait is bounded, and a
      // timeout sets kErrSplitWait in the workspace's error word, which sits
      // right before the counter region.  Each workgroup leaves (and the last
      // resets both counters) before reading, so none can still be waiting
      // when the counters go back to zero.
      if (threadIdx.x == 0) {
        __hip_atomic_fetch_add(cnt, 1 + (foreign ? 1 << (16 + kc) : 0), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        int v = 0;
        for (int it = 0; ((v = __hip_atomic_load(cnt, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) & 0xffff) < nkc; ++it) {
          if (it >= kSplitSpinMax) {
            atomicOr(a.counters - kSplitErrOffset, kErrSplitWait);
            break;
          }
          __builtin_amdgcn_s_sleep(2);
        }
        s_last = (int)((unsigned)v >> 16);  // the foreign chunks
        if (__hip_atomic_fetch_add(cnt + 1, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == nkc - 1) {
          __hip_atomic_store(cnt, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          __hip_atomic_store(cnt + 1, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
      }
      __syncthreads();
      const unsigned fmask = (unsigned)s_last, all = (1u << nkc) - 1u;
      const int valid = min(ROWS, M - m0);
      if (fmask != 0 && fmask != all) {
        // mixed: the first chunk on the expected XCD finishes the block
        if (kc != __builtin_ctz(~fmask & all)) return;
        mhi = m0 + valid;
      } else {
        const int rs = (valid + nkc - 1) / nkc;
        mlo = min(m0 + kc * rs, m0 + valid);
        mhi = min(mlo + rs, m0 + valid);
      }
      for (int j0 = 0; j0 < nkc; j0 += kRedBatch) {
        f32x4 v[kRedBatch][MT];
#pragma unroll
        for (int q = 0; q < kRedBatch; ++q) {
          const int j = min(j0 + q, nkc - 1);
          const bool jl2 = a.par_l2 && !((fmask >> j) & 1u);
#pragma unroll
          for (int mt = 0; mt < MT; ++mt) {
            const int m = m0 + mt * 16 + r;
            v[q][mt] = m >= mlo && m < mhi ? (jl2 ? xcd_load(prs, poff(j, m)) : coherent_load(prs, poff(j, m)))
                                           : f32x4{0.f, 0.f, 0.f, 0.f};
          }
        }
#pragma unroll
        for (int q = 0; q < kRedBatch; ++q)
          if (j0 + q < nkc) {
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) acc[mt] = j0 + q == 0 ? v[q][mt] : acc[mt] + v[q][mt];
          }
      }
    } else {
    if (threadIdx.x == 0)
      s_last = (__hip_atomic_fetch_add(cnt, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == nkc - 1);
    __syncthreads();
    if (!s_last) return;
    if (threadIdx.x == 0) __hip_atomic_store(cnt, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);  // next launch
    // sum all nkc partials (this workgroup's own included, read back) in
    // chunk order; the loads of kRedBatch chunks are issued together (one at
    // a time, each chunk cost a full memory round trip)
    for (int j0 = 0; j0 < nkc; j0 += kRedBatch) {
      f32x4 v[kRedBatch][MT];
#pragma unroll
      for (int q = 0; q < kRedBatch; ++q)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          const int m = min(m0 + mt * 16 + r, M - 1);  // rows past M: read in range, dropped below
          v[q][mt] = coherent_load(prs, poff(min(j0 + q, nkc - 1), m));
        }
#pragma unroll
      for (int q = 0; q < kRedBatch; ++q)
        if (j0 + q < nkc) {
#pragma unroll
          for (int mt = 0; mt < MT; ++mt) acc[mt] = j0 + q == 0 ? v[q][mt] : acc[mt] + v[q][mt];
        }
    }
    }
  }

  if (scaled) {
    // 1/rms of this workgroup's rows: lane sums in order, a 3-step butterfly
    // over the row's 8 lanes (LDS is free: the loop ended on a barrier)
    float t = 0.f;
#pragma unroll
    for (int j = 0; j < 8; ++j) t += ssq_v[j];
    t += __shfl_xor(t, 1);
    t += __shfl_xor(t, 2);
    t += __shfl_xor(t, 4);
    if (threadIdx.x % 8 == 0 && (int)threadIdx.x / 8 < ROWS) s_rinv[threadIdx.x / 8] = 1.0f / sqrtf(t / (float)K + a.eps);
    __syncthreads();
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[mt] *= s_rinv[mt * 16 + r];
  }

  if constexpr (EPI == kEpiSwiglu) {
    // up waves hand their accumulators to the gate waves (LDS is free: the
    // stage loop ended on a barrier)
    f32x4* ex = reinterpret_cast<f32x4*>(&xs[0][0]);
    static_assert(sizeof(xs) >= (size_t)TPW * MT * 64 * sizeof(f32x4), "exchange does not fit");
    if (half == 1) {
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) ex[((wave - TPW) * MT + mt) * 64 + lane] = acc[mt];
    }
    __syncthreads();
    if (half == 1 || !active) return;
    const int n = otile * 16 + 4 * g;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const int m = m0 + mt * 16 + r;
      if (m < mlo || m >= mhi) continue;
      const f32x4 gt = acc[mt], up = ex[(wave * MT + mt) * 64 + lane];
      u32x2 o;
      o[0] = pack_bf16x2(silu_mul(gt[0], up[0]), silu_mul(gt[1], up[1]));
      o[1] = pack_bf16x2(silu_mul(gt[2], up[2]), silu_mul(gt[3], up[3]));
      bf16_t* yp = a.ykbM ? static_cast<bf16_t*>(a.Y) + ((size_t)(n >> 5) * a.ykbM + m) * 32 + (n & 31)
                          : static_cast<bf16_t*>(a.Y) + (size_t)m * Nout + n;
      *reinterpret_cast<u32x2*>(yp) = o;
    }
  } else if constexpr (EPI == kEpiStore || EPI == kEpiLogits) {
    // The MFMA result layout puts 16 rows x 64 bytes in one store
    // instruction; staged through LDS, each wave instead writes two 512-byte
    // row segments per instruction (full cache lines).  LDS is free: the stage
    // loop (or the split-K hand-off) ended on a barrier.
    constexpr int OS = TPW * 16 + 4;  // row stride in floats
    static_assert(sizeof(xs) >= (size_t)ROWS * OS * sizeof(float), "output tile does not fit");
    float* ot = reinterpret_cast<float*>(&xs[0][0]);
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int i = 0; i < 4; ++i) ot[(mt * 16 + r) * OS + wave * 16 + 4 * g + i] = acc[mt][i];
    __syncthreads();
    const int n0 = blockIdx.x * TPW * 16;
    if constexpr (EPI == kEpiLogits) {
      // softmax statistics of this 128-column chunk, 8 lanes per row
      const int row = min((int)threadIdx.x / kStatLanes, ROWS - 1), c = threadIdx.x % kStatLanes;
      float v[kStatPer];
#pragma unroll
      for (int e = 0; e < kStatPer; ++e)
        v[e] = n0 + c * kStatPer + e < Nout ? ot[row * OS + c * kStatPer + e] : -INFINITY;
      float cm, cs;
      chunk_stats(v, cm, cs);
      const int m = m0 + row;
      if (c == 0 && (int)threadIdx.x / kStatLanes < ROWS && m >= mlo && m < mhi) {
        a.stats[((size_t)m * a.nch + blockIdx.x) * 2] = cm;
        a.stats[((size_t)m * a.nch + blockIdx.x) * 2 + 1] = cs;
      }
    }
    constexpr int PIECES = ROWS * TPW * 4;  // 16-byte pieces of the tile
#pragma unroll
    for (int it = 0; it < (PIECES + NTH - 1) / NTH; ++it) {
      const int idx = threadIdx.x + it * NTH;
      const int row = idx / (TPW * 4), c4 = (idx % (TPW * 4)) * 4;
      const int m = m0 + row, n = n0 + c4;
      if (idx < PIECES && m >= mlo && m < mhi && n < Nout)
        *reinterpret_cast<f32x4*>(static_cast<float*>(a.Y) + (size_t)m * Nout + n) =
            *reinterpret_cast<const f32x4*>(&ot[row * OS + c4]);
    }
  } else if constexpr (EPI == kEpiQkvRope) {
    // this workgroup's 128 columns are head hd; rows m0 .. m0+ROWS-1
    constexpr int OS = TPW * 16 + 4;
    static_assert(sizeof(xs) >= (size_t)ROWS * OS * sizeof(float), "output tile does not fit");
    float* ot = reinterpret_cast<float*>(&xs[0][0]);
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int i = 0; i < 4; ++i) ot[(mt * 16 + r) * OS + wave * 16 + 4 * g + i] = acc[mt][i];
    __syncthreads();
    const QkvRope& rp = a.rope;
    const int hd = blockIdx.x, T = rp.T, H = rp.H, Hkv = rp.Hkv;
    const int r_lo = mlo - m0, r_hi = mhi - m0;  // this workgroup's rows of the tile
    if (hd < H + Hkv) {
      bf16_t* base = static_cast<bf16_t*>(hd < H ? rp.q_out : rp.win_k);
#pragma unroll
      for (int it = 0; it < RP_IT; ++it) {
        const int u = threadIdx.x + it * NTH, row = u / 64, j = u % 64, m = m0 + row;
        if (row >= r_hi) break;
        if (row < r_lo) continue;
        const int b = m / T, i = m % T;
        const float cs = __uint_as_float(cs_pre[it][0]), sn = __uint_as_float(cs_pre[it][1]);
        const float x1 = ot[row * OS + j], x2 = ot[row * OS + j + 64];
        bf16_t* dst = hd < H ? base + ((size_t)m * H + hd) * 128
                             : base + (((size_t)b * Hkv + (hd - H)) * kBlock + i) * 128;
        dst[j] = f2bf(x1 * cs - x2 * sn);
        dst[j + 64] = f2bf(x2 * cs + x1 * sn);
      }
      // unused slots T..15 of the K window blocks of the sequences that start here
      if (hd >= H) {
        bf16_t* wb0 = static_cast<bf16_t*>(rp.win_k);
        const int nz = (kBlock - T) * 128 / 8;  // 16-byte pieces
        for (int b = (mlo + T - 1) / T; b * T < mhi; ++b)
          for (int u = threadIdx.x; u < nz; u += NTH)
            *reinterpret_cast<u32x4*>(wb0 + (((size_t)b * Hkv + (hd - H)) * kBlock + T) * 128 + u * 8) =
                u32x4{0u, 0u, 0u, 0u};
      }
    } else {
      // V: one thread per (sequence, head dim) writes the dim's whole 16-slot
      // window row (its T values, then zeros) as two 16-byte stores, for the
      // sequences whose rows all lie in this workgroup (the others' rows are
      // written one value at a time)
      bf16_t* vb = static_cast<bf16_t*>(rp.win_v);
      const int gv = hd - H - Hkv;
      const int b0 = (mlo + T - 1) / T, b1 = mhi / T;  // whole sequences [b0, b1)
      for (int u = threadIdx.x; u < (b1 - b0) * 128; u += NTH) {
        const int b = b0 + u / 128, dd = u % 128;
        uint32_t w[8];
#pragma unroll
        for (int p2 = 0; p2 < 8; ++p2) {
          const int i0 = 2 * p2, i1 = 2 * p2 + 1;
          const float v0 = i0 < T ? ot[(b * T + i0 - m0) * OS + dd] : 0.f;
          const float v1 = i1 < T ? ot[(b * T + i1 - m0) * OS + dd] : 0.f;
          w[p2] = pack_bf16x2(v0, v1);
        }
        u32x4* dst = reinterpret_cast<u32x4*>(vb + (((size_t)b * Hkv + gv) * 128 + dd) * kBlock);
        dst[0] = u32x4{w[0], w[1], w[2], w[3]};
        dst[1] = u32x4{w[4], w[5], w[6], w[7]};
      }
      for (int u = threadIdx.x; u < (r_hi - r_lo) * 128; u += NTH) {  // rows of sequences cut by an edge
        const int row = r_lo + u / 128, dd = u % 128, m = m0 + row, b = m / T, i = m % T;
        if (b >= b0 && b < b1) continue;
        vb[(((size_t)b * Hkv + gv) * 128 + dd) * kBlock + i] = f2bf(ot[row * OS + dd]);
        if (i == 0)
          for (int sl = T; sl < kBlock; ++sl) vb[(((size_t)b * Hkv + gv) * 128 + dd) * kBlock + sl] = 0;
      }
    }
    if (hd == 0 && mlo == 0) {
      const int B = M / T;
      for (int u = threadIdx.x; u < B; u += NTH)
        if (rp.ctx_snap) rp.ctx_snap[u] = rp.ctx[u];
      for (int u = threadIdx.x; u < B * Hkv; u += NTH)
        if (rp.attn_cnt) rp.attn_cnt[u * kCounterStride] = 0;
    }
  } else if constexpr (EPI == kEpiResidualNorm) {
    // h += acc through an LDS-staged tile, 32 lanes per 512-byte row segment;
    // each row segment also yields bf16(h * gain) and its sum of h^2 (lane
    // order, then a 5-step butterfly over the 32 lanes)
    constexpr int OS = TPW * 16 + 4;
    static_assert(sizeof(xs) >= (size_t)ROWS * OS * sizeof(float), "output tile does not fit");
    float* ot = reinterpret_cast<float*>(&xs[0][0]);
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int i = 0; i < 4; ++i) ot[(mt * 16 + r) * OS + wave * 16 + 4 * g + i] = acc[mt][i];
    __syncthreads();
    const int n0 = blockIdx.x * TPW * 16;
    constexpr int PIECES = RN_PIECES;
    static_assert(PIECES % NTH == 0 || PIECES < NTH, "row segments must not straddle passes");
#pragma unroll
    for (int it = 0; it < RN_IT; ++it) {
      const int idx = threadIdx.x + it * NTH;
      const int row = idx / (TPW * 4), c4 = (idx % (TPW * 4)) * 4;
      const int m = m0 + row, n = n0 + c4;
      float part = 0.f;
      const bool ok = idx < PIECES && m >= mlo && m < mhi && n < Nout;
      if (ok) {
        f32x4* hp = reinterpret_cast<f32x4*>(static_cast<float*>(a.Y) + (size_t)m * Nout + n);
        const f32x4 hv = h_pre[it] + *reinterpret_cast<const f32x4*>(&ot[row * OS + c4]);
        *hp = hv;
        const u32x2 gw = g_pre[it];
        u32x2 o;
        o[0] = pack_bf16x2(hv[0] * bf2f((bf16_t)(gw[0] & 0xffffu)), hv[1] * bf2f((bf16_t)(gw[0] >> 16)));
        o[1] = pack_bf16x2(hv[2] * bf2f((bf16_t)(gw[1] & 0xffffu)), hv[3] * bf2f((bf16_t)(gw[1] >> 16)));
        *reinterpret_cast<u32x2*>(a.xg_kb ? a.xg + ((size_t)(n >> 5) * M + m) * 32 + (n & 31) : a.xg + (size_t)m * Nout + n) = o;
        part = hv[0] * hv[0];
        part = fmaf(hv[1], hv[1], part);
        part = fmaf(hv[2], hv[2], part);
        part = fmaf(hv[3], hv[3], part);
      }
      part += __shfl_xor(part, 1);
      part += __shfl_xor(part, 2);
      part += __shfl_xor(part, 4);
      part += __shfl_xor(part, 8);
      part += __shfl_xor(part, 16);
      if ((idx % (TPW * 4)) == 0 && idx < PIECES && m >= mlo && m < mhi) a.ssq_out[(size_t)m * a.nch + blockIdx.x] = part;
    }
  } else {
    if (!active) return;
    const int n = otile * 16 + 4 * g;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const int m = m0 + mt * 16 + r;
      if (m < mlo || m >= mhi) continue;
      f32x4* p = reinterpret_cast<f32x4*>(static_cast<float*>(a.Y) + (size_t)m * Nout + n);
      *p = *p + acc[mt];
    }
  }
}

// LM head (and other wide fp32-store GEMMs) for windows of up to 96 rows: a
// persistent form of the streaming kernel.  Logits stores issued while the
// weight stream runs cost far more than their bytes (the HBM keeps turning the
// bus around between reads and writes), so each workgroup streams
// kLogitsTiles groups of NW * 16 weight rows (one row tile per wave; one group
// for windows of more than 64 rows) one after another, keeps each finished logits tile in registers, and writes them all
// after its last group (through one LDS tile, as full row segments).  Softmax statistics (skipped when stats is null): the
// (max, sum of exp) of each 128-column chunk of its groups, merged per row in
// a fixed order into one pair per workgroup, stats[row][blockIdx.x] -- so the
// acceptance reads one pair per workgroup and row, not one per chunk.
// Row scale (folded RMSNorm) and statistics as in the kEpiLogits epilogue of
// gemm_stream_kernel.
constexpr int kLogitsTiles = 2;
constexpr int kLogitsMaxTiles = 6;  // 16-row tiles of the largest window it takes
// groups per workgroup of an MT-row window: windows of more than 64 rows keep
// one finished group in registers (two would not fit beside the stream's)
constexpr int logits_tiles(int mt) { return mt > 4 ? 1 : kLogitsTiles; }
// Waves per workgroup for windows of more than 16 rows: 256 weight rows per
// group, so each staged x stage feeds 16 waves (with 8, the x traffic of a
// 48-row window is 37% of the weight traffic and holds the kernel ~4% below
// the read rate it reaches at 16 rows).
constexpr int kLogitsWaves = 16;
template <int MT, int NW>
__global__ __launch_bounds__(NW * 64) void gemm_logits_kernel(GemmK a) {
  constexpr int TPW = NW;                // 16-column output tiles per group
  constexpr int CPG = TPW * 16 / kStatChunk;  // statistics chunks per group
  static_assert(CPG * kStatChunk == TPW * 16, "a group's columns are whole statistics chunks");
  constexpr int ROWS = MT * 16, NTH = NW * 64;
  static_assert(ROWS * 8 <= NTH, "one pass of sum-of-squares lanes");
  constexpr int CH = ROWS * (kSK / 8), PT = (CH + NTH - 1) / NTH;
  constexpr int OS = TPW * 16 + 4;  // LDS row stride of an output tile, in floats
  __shared__ __attribute__((aligned(16))) bf16_t xs[2][ROWS * kXStride];
  __shared__ __attribute__((aligned(16))) float ot[ROWS * OS];
  __shared__ float s_rinv[ROWS];
  constexpr int LT = logits_tiles(MT);
  __shared__ float2 s_cst[LT][ROWS * CPG];  // chunk statistics of each group

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r = lane & 15, g = lane >> 4;
  const int M = a.M, Nout = a.Nout, K = a.K, KS = a.KS;
  const int nto = Nout / 16, ngroups = (nto + TPW - 1) / TPW;
  const int nst = (KS + kSU - 1) / kSU;

  const bf16_t* xp[PT];
  int xo[PT], xc[PT];
#pragma unroll
  for (int c = 0; c < PT; ++c) {
    const int idx = min((int)threadIdx.x + c * NTH, CH - 1);
    const int row = idx / (kSK / 8), col = (idx % (kSK / 8)) * 8;
    xp[c] = a.X + (size_t)min(row, M - 1) * K;
    xc[c] = col;
    xo[c] = row * kXStride + col;
  }
  const bool scaled = a.ssq_in != nullptr;
  float ssq_v[8];
  if (scaled) {
    const int row = min((int)threadIdx.x / 8, ROWS - 1), c = threadIdx.x % 8;
    const float* sp = a.ssq_in + (size_t)min(row, M - 1) * a.nt_in;
#pragma unroll
    for (int j = 0; j < 8; ++j) ssq_v[j] = c + 8 * j < a.nt_in ? sp[c + 8 * j] : 0.f;
  }
  auto row_scales = [&] {  // 1/rms of every row into s_rinv
    float t = 0.f;
#pragma unroll
    for (int j = 0; j < 8; ++j) t += ssq_v[j];
    t += __shfl_xor(t, 1);
    t += __shfl_xor(t, 2);
    t += __shfl_xor(t, 4);
    if (threadIdx.x % 8 == 0 && (int)threadIdx.x / 8 < ROWS) s_rinv[threadIdx.x / 8] = 1.0f / sqrtf(t / (float)K + a.eps);
    __syncthreads();
  };
  // Windows of more than 64 rows have no registers to spare for the partials
  // across the weight stream: their scales are taken before it.
  if (MT > 4 && scaled) row_scales();

  // The finished tiles stay in registers (tile tt in fin[tt]) until the last
  // group's weights have been streamed; then each passes through the one LDS
  // output tile for its statistics and its row-segment stores.
  static_assert(LT == 1 || LT == 2, "finished tiles are held in one or two register sets");
  f32x4 fin0[MT], fin1[LT == 2 ? MT : 1];
  int done = 0;
  for (int tt = 0; tt < LT; ++tt) {
    const int grp = blockIdx.x + tt * gridDim.x;
    if (grp >= ngroups) break;
    const int wtile = min(grp * TPW + wave, nto - 1);
    const bf16_t* wp = a.W + ((size_t)(wtile >> 3) * KS * 8 + (wtile & 7)) * 512 + lane * 8;
    f32x4 acc[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
    stream_tile<MT, 2, PT>(acc, wp, xp, xc, xo, K, KS, 0, nst, &xs[0][0]);
    if (scaled) {
      if (MT <= 4 && tt == 0) row_scales();
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) acc[mt] *= s_rinv[mt * 16 + r];
    }
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      if (tt == 0) fin0[mt] = acc[mt];
      else if constexpr (LT == 2) fin1[mt] = acc[mt];
    }
    done = tt + 1;
  }
  constexpr int PIECES = ROWS * TPW * 4;
  for (int tt = 0; tt < done; ++tt) {
    const int grp = blockIdx.x + tt * gridDim.x;
    __syncthreads();  // the previous tile's stores have read the LDS tile
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int i = 0; i < 4; ++i) ot[(mt * 16 + r) * OS + wave * 16 + 4 * g + i] = tt == 0 ? fin0[mt][i] : fin1[LT == 2 ? mt : 0][i];
    __syncthreads();
    // the finished tile, full 512-byte row segments (issued first: the
    // statistics below only read LDS and run while the stores drain)
    const int n0 = grp * TPW * 16;
#pragma unroll
    for (int it = 0; it < (PIECES + NTH - 1) / NTH; ++it) {
      const int idx = threadIdx.x + it * NTH;
      const int row = idx / (TPW * 4), c4 = (idx % (TPW * 4)) * 4;
      const int n = n0 + c4;
      if (idx < PIECES && row < M && n < Nout)
        *reinterpret_cast<f32x4*>(static_cast<float*>(a.Y) + (size_t)row * Nout + n) =
            *reinterpret_cast<const f32x4*>(&ot[row * OS + c4]);
    }
    if (a.stats) {  // softmax statistics of the group's chunks, 8 lanes per (row, chunk)
      const int c = threadIdx.x % kStatLanes;
      for (int unit = threadIdx.x / kStatLanes; unit < ROWS * CPG; unit += NTH / kStatLanes) {
        const int row = unit / CPG, ch = unit % CPG;
        const int c0 = n0 + ch * kStatChunk;
        float v[kStatPer];
#pragma unroll
        for (int e = 0; e < kStatPer; ++e)
          v[e] = c0 + c * kStatPer + e < Nout ? ot[row * OS + ch * kStatChunk + c * kStatPer + e] : -INFINITY;
        float cm, cs;
        chunk_stats(v, cm, cs);
        if (c == 0) s_cst[tt][unit] = float2{cm, cs};
      }
    }
  }
  if (a.stats) {  // one (max, sum) per row: the chunks merged in (group, chunk) order
    __syncthreads();
    const int row = threadIdx.x;
    if (row < ROWS && row < M) {
      float m = -INFINITY, sum = 0.f;
      for (int tt = 0; tt < done; ++tt)
#pragma unroll
        for (int ch = 0; ch < CPG; ++ch) {
          const float2 c2 = s_cst[tt][row * CPG + ch];
          if (c2.x == -INFINITY) continue;
          if (m == -INFINITY) {
            m = c2.x;
            sum = c2.y;
          } else if (c2.x > m) {
            sum = sum * expf(m - c2.x) + c2.y;
            m = c2.x;
          } else {
            sum += c2.y * expf(c2.x - m);
          }
        }
      *reinterpret_cast<float2*>(a.stats + ((size_t)row * a.nch + blockIdx.x) * 2) = float2{m, sum};
    }
  }
}

// Packed weight layout: element (n, k) of a [N][K] row-major matrix goes to
//   ((((n / 128) * (K / 32) + k / 32) * 8 + (n / 16) % 8) * 64 + ((k % 32) / 8) * 16 + n % 16) * 8 + k % 8
// Rows past N up to the next multiple of 128 are zero.  One thread per
// 16-byte destination piece.
__global__ __launch_bounds__(256) void pack_weight_kernel(const bf16_t* __restrict__ src, bf16_t* __restrict__ dst,
                                                          int N, int K, size_t pieces) {
  const int KS = K / 32;
  for (size_t p = (size_t)blockIdx.x * 256 + threadIdx.x; p < pieces; p += (size_t)gridDim.x * 256) {
    const int lane = (int)(p & 63), t = (int)((p >> 6) & 7);
    const size_t q = p >> 9;
    const int ks = (int)(q % KS);
    const size_t grp = q / KS;
    const size_t n = grp * 128 + t * 16 + (lane & 15);
    const int k = ks * 32 + (lane >> 4) * 8;
    u32x4 v = u32x4{0u, 0u, 0u, 0u};
    if (n < (size_t)N) v = *reinterpret_cast<const u32x4*>(src + n * K + k);
    *reinterpret_cast<u32x4*>(dst + p * 8) = v;
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

template <int EPI, int NB>
hipError_t launch_stream_nb(const GemmK& a0, const GemmPlan& p, hipStream_t s) {
  const dim3 grid(p.ntiles, p.mblocks, p.nkc), block(kNW * 64);
  GemmK a = a0;
  a.par = p.par && p.nkc > 1 && (long)p.ntiles * p.mblocks * p.nkc <= device_cus() ? 1 : 0;
  // chunks kc of block (t, mb) are workgroups t + ntiles (mb + mblocks kc):
  // one XCD under round-robin dispatch when ntiles * mblocks is a multiple of 8
  a.par_l2 = a.par && p.nkc <= kSplitL2MaxChunks && ((long)p.ntiles * p.mblocks) % 8 == 0 ? 1 : 0;
  a.foreign = split_foreign_mask();
  switch (p.mt) {
    case 1: hipLaunchKernelGGL((gemm_stream_kernel<1, EPI, NB>), grid, block, 0, s, a); break;
    case 2: hipLaunchKernelGGL((gemm_stream_kernel<2, EPI, NB>), grid, block, 0, s, a); break;
    case 3: hipLaunchKernelGGL((gemm_stream_kernel<3, EPI, NB>), grid, block, 0, s, a); break;
    default: hipLaunchKernelGGL((gemm_stream_kernel<4, EPI, NB>), grid, block, 0, s, a); break;
  }
  return hipGetLastError();
}

template <int EPI>
hipError_t launch_stream(const GemmK& a, const GemmPlan& p, hipStream_t s) {
  if (p.mt > 4) return hipErrorInvalidValue;  // 5 and 6 row tiles: the persistent kernel only
  return p.depth >= 3 ? launch_stream_nb<EPI, 4>(a, p, s) : launch_stream_nb<EPI, 2>(a, p, s);
}

// The LM head: the persistent kernel when the window fits one 48-row block and
// K is not split (its grid size: the statistics pairs per row), else 0 and the
// streaming kernel's kEpiLogits epilogue.
int logits_persistent_grid(const GemmPlan& p, int Nout) {
  if (p.nkc > 1 || p.mblocks > 1 || p.mt > kLogitsMaxTiles || p.depth >= 3) return 0;
  // 16-row windows stage little x per weight byte: 8 waves per workgroup
  const int NW = p.mt == 1 ? kNW : kLogitsWaves;
  const int groups = (Nout / 16 + NW - 1) / NW;
  const int lt = logits_tiles(p.mt);
  return (groups + lt - 1) / lt;
}

hipError_t launch_logits(const GemmK& a, const GemmPlan& p, hipStream_t s) {
  const int pg = logits_persistent_grid(p, a.Nout);
  if (pg == 0) return a.stats ? launch_stream<kEpiLogits>(a, p, s) : launch_stream<kEpiStore>(a, p, s);
  const int NW = p.mt == 1 ? kNW : kLogitsWaves;
  const dim3 grid(pg), block(NW * 64);
  switch (p.mt) {
    case 1: hipLaunchKernelGGL((gemm_logits_kernel<1, kNW>), grid, block, 0, s, a); break;
    case 2: hipLaunchKernelGGL((gemm_logits_kernel<2, kLogitsWaves>), grid, block, 0, s, a); break;
    case 3: hipLaunchKernelGGL((gemm_logits_kernel<3, kLogitsWaves>), grid, block, 0, s, a); break;
    case 4: hipLaunchKernelGGL((gemm_logits_kernel<4, kLogitsWaves>), grid, block, 0, s, a); break;
    case 5: hipLaunchKernelGGL((gemm_logits_kernel<5, kLogitsWaves>), grid, block, 0, s, a); break;
    default: hipLaunchKernelGGL((gemm_logits_kernel<6, kLogitsWaves>), grid, block, 0, s, a); break;
  }
  return hipGetLastError();
}

}  // namespace

static size_t al256(size_t x) { return (x + 255) & ~(size_t)255; }

namespace {
// Buffers of a stream-K schedule: the most segments any tile is cut into
// (partials: that many M x N fp32 copies) and one counter per workgroup.
void tile_sk_buffers(GemmPlan& p, int M, int N, int K) {
  const long KU = K / 64, U = (long)p.ntiles * KU, GS = p.grid / p.mblocks;
  auto owner = [&](long X) { return ((X + 1) * GS + U - 1) / U - 1; };
  long smax = 1;
  for (long t = 0; t < p.ntiles; ++t) smax = std::max(smax, owner(t * KU + KU - 1) - owner(t * KU) + 1);
  p.nkc = (int)smax;
  p.part_bytes = smax > 1 ? al256((size_t)smax * M * N * 4) : 0;
  p.counter_bytes = smax > 1 ? al256((size_t)p.grid * kCounterStride * 4) : 0;
}
}  // namespace

unsigned split_foreign_mask() {
  static const unsigned mask = [] {
    const char* e = getenv("NJ_TEST_SPLIT_FOREIGN");
    return e ? (unsigned)strtoul(e, nullptr, 0) : 0u;
  }();
  return mask;
}

int device_cus() {
  static const int cus = [] {
    int dev = 0, n = 0;
    if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
      return 0;
    return n;
  }();
  return cus;
}

GemmPlan gemm_tile_plan_sk(int M, int N, int K, int epi, int tile, int grid) {
  GemmPlan p{};
  const int NG = epi == kEpiSwiglu ? 2 : 1;
  const int Nout = N / NG;
  p.tile = tile;
  const int bm = tile_bm(tile), bno = tile_bn(tile) / NG;
  p.mblocks = (M + bm - 1) / bm;
  p.ntiles = (Nout + bno - 1) / bno;
  // shares per M tile: the grid rounded down to a multiple of the M tiles
  const long units = (long)p.ntiles * (K / 64);
  const long shares = std::max(1L, std::min({(long)grid / p.mblocks, units, ((1L << 20) - 1) / p.mblocks}));
  p.grid = (int)(shares * p.mblocks);
  p.stages_per_chunk = (int)((units + shares - 1) / shares);  // units per workgroup, at most
  p.depth = 1;
  tile_sk_buffers(p, M, N, K);
  p.par = p.nkc > 1 && p.grid <= kParMaxGrid && tile_one_segment(p, K) ? 1 : 0;
  return p;
}

GemmPlan gemm_tile_plan(int M, int N, int K, int epi, int tile, int nkc) {
  const int NG = epi == kEpiSwiglu ? 2 : 1;
  const int tiles = ((M + tile_bm(tile) - 1) / tile_bm(tile)) * ((N / NG + tile_bn(tile) / NG - 1) / (tile_bn(tile) / NG));
  return gemm_tile_plan_sk(M, N, K, epi, tile, tiles * std::max(1, std::min(nkc, K / 64)));
}

namespace {
// Cost models (seconds) used to pick the kernel for windows of 65+ rows,
// with constants fitted to sweeps of the 8B- and 7B-shaped GEMMs (QKV, O,
// gate/up, down, LM head) at 65..2048 rows over both kernels, every tile
// shape, K splits of 1..8 (slice-reduced) and a 256-workgroup stream-K grid:
// the plan chosen is the fastest measured one, or within 3% of it, at 70 of
// 83 points and within 15% at the others (the sustained fractions below are
// fitted for ranking plans, so they sit above the measured ones).
// Tiled kernel: rounds of resident workgroups times one tile's MFMA time at
// the tile shape's sustained fraction of peak, plus, when tiles are cut, the
// last arriver's reduction (one CU reads nkc partial tiles) and the partial
// traffic.
constexpr double kLaunch = 5e-6;
constexpr double kParFixed = 3e-6;  // the wait for a tile's slowest workgroup and the departure
constexpr double kCuPeak = 2.5e15 / 256.0;  // bf16 MFMA FLOP/s of one CU
constexpr int kTileShapes[] = {kTile256x256, kTile192x256, kTile160x256, kTile128x256, kTile96x256, kTile96x128,
                               kTile128x128};
// sustained fraction of a CU's MFMA peak with k-blocked x
double tile_eff(int tile) {
  switch (tile) {
    case kTile256x256: return 0.64;
    case kTile192x256:
    case kTile160x256: return 0.58;
    case kTile128x256: return 0.50;
    case kTile96x256: return 0.40;
    default: return 0.32;  // 96 x 128 and 128 x 128
  }
}
// workgroups of the shape a CU holds at once (LDS and registers): two of the
// small tiles, one of the others
int tile_occupancy(int tile) { return tile == kTile128x128 || tile == kTile96x128 ? 2 : 1; }
double tile_cost(const GemmPlan& p, int M, int N, int K) {
  const int bm = tile_bm(p.tile), bn = tile_bn(p.tile);
  const double wgs = (double)p.grid;
  // a CU takes a second workgroup only when the grid has more than one per CU
  const double per_cu = std::max(1.0, std::min((double)tile_occupancy(p.tile), std::ceil(wgs / 256.0)));
  const double rounds = std::ceil(wgs / (256.0 * per_cu));
  double t = rounds * per_cu * 2.0 * bm * bn * (64.0 * p.stages_per_chunk) / (kCuPeak * tile_eff(p.tile));
  if (p.nkc > 1) {
    // cut tiles: one CU reads the nkc partial tiles (last arriver), or, with
    // the slice reduction, each of the nkc workgroups reads one tile's worth
    t += (p.par ? kParFixed + bm * bn * 4 / 1e11 : 2.0 * p.nkc * bm * bn * 4 / 5e10) +
         2.0 * p.nkc * (double)M * N * 4 / 5e12;
  }
  return t + kLaunch;
}
// Weight-streaming kernel: rounds of workgroups (one per CU), each streaming
// 128 weight rows of its K chunk at ~40 GB/s per CU or multiplying them by
// its 16..64 x rows at ~0.22 of the CU's MFMA peak (LDS-bound), whichever is
// longer.
double stream_cost(int M, int N, int K, int epi) {
  const GemmPlan p = gemm_stream_plan(M, N, K, epi, 0, 1);
  const double rounds = std::ceil((double)p.ntiles * p.mblocks * p.nkc / 256.0);
  const double kchunk = 128.0 * p.stages_per_chunk;
  const double t_wg = std::max(128.0 * kchunk * 2 / 40e9, 2.0 * 128 * (16.0 * p.mt) * kchunk / (kCuPeak * 0.22));
  return 8e-6 + rounds * t_wg + (p.nkc > 1 ? 3e-6 : 0.0);
}
// A QKV projection that streams applies RoPE and stores the window K/V in its
// epilogue; a tiled one leaves that to a kernel of its own.
double rope_kernel_cost(int M) { return 5e-6 + 9e-9 * M; }
}  // namespace

GemmPlan gemm_tile_choose(int M, int N, int K, int epi, int only_tile) {
  GemmPlan best{};
  double bc = 1e30;
  auto consider = [&](const GemmPlan& p) {
    if (p.nkc > 1 && (p.counter_bytes > kGemmCounterBytes || p.part_bytes > kSplitPartCap)) return;
    const double c = tile_cost(p, M, N, K);
    if (c < bc) bc = c, best = p;
  };
  for (int tile : kTileShapes) {
    if (only_tile != kTileNone && tile != only_tile) continue;
    for (int nkc = 1; nkc <= 8; nkc *= 2) {
      if (nkc > 1 && K / 64 / nkc < 8) break;
      consider(gemm_tile_plan(M, N, K, epi, tile, nkc));
    }
    // Stream-K on one workgroup per CU when the tiles leave CUs idle (not for
    // the 256 x 256 tile, which runs one segment per workgroup).
    if (tile != kTile256x256 && (long)gemm_tile_plan(M, N, K, epi, tile, 1).grid % 256 != 0)
      consider(gemm_tile_plan_sk(M, N, K, epi, tile, 256));
  }
  return best;
}

bool tile_fits(int M, int N, int K) {
  return K % 64 == 0 && (long)M * K < (1L << 31) && (long)packed_weight_elems(N, K) < (1L << 31);
}

GemmPlan gemm_logits_widen(const GemmPlan& p, int M, int N) {
  if (p.tile != kTileNone || p.nkc > 1 || p.depth >= 3 || M <= 64 || M > 16 * kLogitsMaxTiles) return p;
  GemmPlan q = p;
  q.mt = (M + 15) / 16;
  q.mblocks = 1;
  return logits_persistent_grid(q, N) > 0 ? q : p;
}

namespace {
GemmPlan gemm_plan_uncached(int M, int N, int K, int epi) {
  if (M >= kTileMinRows && tile_fits(M, N, K)) {
    // wide fp32-store GEMMs (the LM head) of up to 96 rows: the persistent
    // kernel reads the weights once and runs ~10% ahead of the best tile
    // (128x256) at 72..96 rows when it fills the chip
    if (epi == kEpiStore) {
      const GemmPlan sp = gemm_logits_widen(gemm_stream_plan(M, N, K, epi, 0, 1), M, N);
      if (sp.mt > 4 && logits_persistent_grid(sp, N) >= 256) return sp;
    }
    const GemmPlan t = gemm_tile_choose(M, N, K, epi, kTileNone);
    const double extra = epi == kEpiQkvRope ? rope_kernel_cost(M) : 0.0;
    if (tile_cost(t, M, N, K) + extra < stream_cost(M, N, K, epi)) return t;
  }
  return gemm_stream_plan(M, N, K, epi, 0, 1);
}
}  // namespace

// The plan depends only on (M, N, K, epilogue) and a verify step asks for
// the same few plans several times per launch (workspace layout, which
// kernels the norms fold into, the launches), while scoring every tile shape
// and stream-K grid costs tens of microseconds of host time for the LM head:
// plans are kept in a small table (cleared when it fills).
GemmPlan gemm_plan(int M, int N, int K, int epi) {
  static std::mutex mu;
  static std::unordered_map<uint64_t, GemmPlan> memo;
  const uint64_t key = ((uint64_t)(uint32_t)M << 40) ^ ((uint64_t)(uint32_t)N << 20) ^ ((uint64_t)(uint32_t)K << 4) ^
                       (uint64_t)(uint32_t)epi;
  {
    std::lock_guard<std::mutex> g(mu);
    const auto it = memo.find(key);
    if (it != memo.end() && it->second.key_m == M && it->second.key_n == N && it->second.key_k == K &&
        it->second.key_epi == epi)
      return it->second;
  }
  GemmPlan p = gemm_plan_uncached(M, N, K, epi);
  p.key_m = M, p.key_n = N, p.key_k = K, p.key_epi = epi;
  std::lock_guard<std::mutex> g(mu);
  if (memo.size() >= 4096) memo.clear();
  memo[key] = p;
  return p;
}

GemmPlan gemm_stream_plan(int M, int N, int K, int epi, int split, int depth) {
  GemmPlan p{};
  p.tile = kTileNone;
  const int NG = epi == kEpiSwiglu ? 2 : 1;
  const int Nout = N / NG;
  p.mt = M >= 64 ? 4 : (M + 15) / 16;
  p.mblocks = (M + p.mt * 16 - 1) / (p.mt * 16);
  p.nw = kNW;
  p.ntiles = (Nout / 16 + kNW / NG - 1) / (kNW / NG);
  const int nst = (K / 32 + kSU - 1) / kSU;
  const long base = (long)p.ntiles * p.mblocks;
  // Split K until ~256 workgroups run, keeping >= 8 stages (1024 k) per chunk
  // so that the x staging and the partial hand-off are amortised.
  int nkc = 1;
  if (split > 0) nkc = std::min(split, nst);
  else
    while (base * nkc * 2 <= kSplitTargetWorkgroups && nst / (nkc * 2) >= 8) nkc *= 2;
  if (split <= 0)
    while (nkc > 1 && (size_t)nkc * M * N * 4 > kSplitPartCap) nkc /= 2;
  p.stages_per_chunk = (nst + nkc - 1) / nkc;
  p.nkc = (nst + p.stages_per_chunk - 1) / p.stages_per_chunk;
  p.depth = depth;
  p.part_bytes = p.nkc > 1 ? al256((size_t)p.nkc * M * N * 4) : 0;
  p.counter_bytes = p.nkc > 1 ? al256((size_t)p.ntiles * p.mblocks * kCounterStride * 4) : 0;
  p.par = p.nkc > 1 && (long)p.ntiles * p.mblocks * p.nkc <= kParMaxGrid ? 1 : 0;
  static_assert(kSplitTargetWorkgroups / 2 * kCounterStride * 4 <= kGemmCounterBytes, "counter region too small");
  return p;
}

hipError_t launch_gemm_plan(const void* x, const void* w, void* y, int M, int N, int K, int epi, const GemmPlan& p,
                            int* counters, float* part, hipStream_t s, bool x_kblocked, bool y_kblocked) {
  if (p.tile != kTileNone)
    return launch_gemm_tile(x, w, y, M, N, K, epi, p, counters, part, s, nullptr, x_kblocked, y_kblocked);
  if (x_kblocked) return hipErrorInvalidValue;  // the streaming kernel reads row-major x
  const int Nout = (epi == kEpiSwiglu) ? N / 2 : N;
  GemmK a{static_cast<const bf16_t*>(x), static_cast<const bf16_t*>(w), y, p.nkc > 1 ? part : nullptr,
          p.nkc > 1 ? counters : nullptr, M, Nout, K, K / 32, p.stages_per_chunk, (int)p.part_bytes, nullptr, 0, nullptr, 0, 0.f, nullptr, nullptr, nullptr, {},
          y_kblocked ? M : 0};
  if (epi == kEpiStore) return launch_logits(a, p, s);  // stats == nullptr: plain store
  if (epi == kEpiResidual) return launch_stream<kEpiResidual>(a, p, s);
  return launch_stream<kEpiSwiglu>(a, p, s);
}

hipError_t launch_gemm_logits(const void* x, const void* w, float* y, float* stats, int M, int N, int K,
                              int* counters, float* part, hipStream_t s, bool* stats_written, bool x_kblocked) {
  const GemmPlan p = gemm_plan(M, N, K, kEpiStore);
  *stats_written = true;
  if (p.tile != kTileNone)
    return launch_gemm_tile(x, w, y, M, N, K, kEpiStore, p, counters, part, s, stats, x_kblocked);
  if (x_kblocked) return hipErrorInvalidValue;  // the streaming kernel reads row-major x
  GemmK a{static_cast<const bf16_t*>(x), static_cast<const bf16_t*>(w), y, p.nkc > 1 ? part : nullptr,
          p.nkc > 1 ? counters : nullptr, M, N, K, K / 32, p.stages_per_chunk, (int)p.part_bytes, stats,
          (N + kStatChunk - 1) / kStatChunk, nullptr, 0, 0.f, nullptr, nullptr, nullptr, {}};
  return launch_logits(a, p, s);
}

bool gemm_streams(int M, int N, int K, int epi) { return gemm_plan(M, N, K, epi).tile == kTileNone; }

int logits_stat_entries(int M, int N, int K) {
  const GemmPlan p = gemm_plan(M, N, K, kEpiStore);
  if (p.tile != kTileNone) return p.ntiles;  // one pair per column tile
  const int pg = logits_persistent_grid(p, N);
  return pg > 0 ? pg : (N + kStatChunk - 1) / kStatChunk;
}

hipError_t launch_gemm_norm(const void* x, const void* w, void* y, int M, int N, int K, int epi, const GemmNorm& nm,
                            int* counters, float* part, hipStream_t s, const QkvRope* rope, bool x_kblocked,
                            bool y_kblocked) {
  const int pe = epi == kEpiResidualNorm ? kEpiResidual : epi == kEpiLogits ? kEpiStore : epi;
  const GemmPlan p = gemm_plan(M, N, K, epi == kEpiQkvRope ? kEpiQkvRope : pe);
  if (p.tile != kTileNone) {
    // the tiled kernel: the row scale in every epilogue, the next norm's
    // inputs from the slice-reduced residual epilogue (it checks the plan);
    // RoPE lives in the streaming epilogue only
    if (epi == kEpiQkvRope) return hipErrorInvalidValue;
    return launch_gemm_tile(x, w, y, M, N, K, pe, p, counters, part, s, epi == kEpiLogits ? nm.stats : nullptr,
                            x_kblocked, y_kblocked, &nm);
  }
  if (x_kblocked) return hipErrorInvalidValue;  // the streaming kernel reads row-major x
  const int Nout = (epi == kEpiSwiglu) ? N / 2 : N;
  GemmK a{static_cast<const bf16_t*>(x), static_cast<const bf16_t*>(w), y, p.nkc > 1 ? part : nullptr,
          p.nkc > 1 ? counters : nullptr, M, Nout, K, K / 32, p.stages_per_chunk, (int)p.part_bytes, nm.stats,
          (Nout + kStatChunk - 1) / kStatChunk, nm.ssq_in, nm.nt_in, nm.eps,
          static_cast<const bf16_t*>(nm.gain), static_cast<bf16_t*>(nm.xg), nm.ssq_out, rope ? *rope : QkvRope{}};
  a.ykbM = y_kblocked ? M : 0;
  a.xg_kb = nm.xg_kb;
  switch (epi) {
    case kEpiQkvRope: return launch_stream<kEpiQkvRope>(a, p, s);
    case kEpiStore: return launch_stream<kEpiStore>(a, p, s);
    case kEpiSwiglu: return launch_stream<kEpiSwiglu>(a, p, s);
    case kEpiLogits: return launch_logits(a, p, s);
    case kEpiResidualNorm: return launch_stream<kEpiResidualNorm>(a, p, s);
    default: return launch_stream<kEpiResidual>(a, p, s);
  }
}

size_t packed_weight_elems(int N, int K) { return (size_t)((N + 127) / 128) * 128 * (size_t)K; }

hipError_t launch_pack_weight(const void* src, void* dst, int N, int K, hipStream_t s) {
  const size_t pieces = packed_weight_elems(N, K) / 8;
  const int grid = (int)std::min<size_t>((pieces + 255) / 256, 65536);
  hipLaunchKernelGGL(pack_weight_kernel, dim3(grid), dim3(256), 0, s, static_cast<const bf16_t*>(src),
                     static_cast<bf16_t*>(dst), N, K, pieces);
  return hipGetLastError();
}

hipError_t launch_gemm(int dtype, const void* x, const void* w, void* y, int M, int N, int K, int epi,
                       int* counters, float* part, hipStream_t s, bool x_kblocked, bool y_kblocked) {
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
  return launch_gemm_plan(x, w, y, M, N, K, epi, gemm_plan(M, N, K, epi), counters, part, s, x_kblocked, y_kblocked);
}

}  // namespace nj
