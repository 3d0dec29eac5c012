// Large-window GEMMs (M = B*(k+1) in the hundreds or thousands): y = x . w^T
// with both operands staged through LDS.
//
// Above M ~ 300 rows the verify step's GEMMs are bound by the matrix cores
// (2*M FLOP per weight byte against a 312 FLOP/byte ridge), so the
// weight-streaming kernel, which re-reads the weights once per 64 window rows
// and feeds every MFMA with one LDS read, is the wrong shape.  Here a
// workgroup owns a BM x BN output tile (x rows x weight rows) and each wave
// multiplies a (BM/WM) x (BN/WN) sub-tile with 16x16x32 bf16 MFMAs, so every
// LDS fragment read feeds TN (or TM) MFMAs.
//
// - Operands go from memory straight into LDS (global_load_lds_dwordx4: no
//   staging registers, no LDS write instructions), one 32-wide k-step per
//   stage, NBUF stage buffers, NBUF-1 stages in flight.  Each stage holds
//   1 KB units of 16 rows x 32 k in MFMA operand order (lane l: row l % 16,
//   k 8 (l / 16) .. +8): a unit is one load instruction (lane l's 16 bytes land
//   at byte 16 l) and one conflict-free fragment read.  Weight units are the
//   packed layout's tiles copied as they are; x units gather 16 row segments.
// - Tile order is XCD-aware: workgroup IDs go round-robin over the 8 XCDs, so
//   the linear ID is remapped to give each XCD a contiguous run of tiles, with
//   the M tiles of one weight tile adjacent.  The weight tile is then fetched
//   from HBM once and re-read by its neighbours from that XCD's L2.
// - Work is scheduled stream-K: the tiles x K/64 units go to the grid's
//   workgroups in equal contiguous shares, so a tile count that does not
//   divide the chip still keeps every CU busy to the end; a tile cut between
//   workgroups is summed in k order by the last to arrive (fixed order, as
//   in the weight-streaming kernel's split K).  A plain K split (or none) is
//   the special case grid = tiles x c.
// - Epilogues as in the weight-streaming kernel: fp32 store, fp32 residual
//   add, and SwiGLU, for which the first half of the weight tile holds gate
//   rows and the second half the matching up rows.
#include "common.h"
#include "kernels.h"
#include <utility>

namespace nj {
namespace {


__device__ __forceinline__ float silu_mul(float gte, float up) { return gte / (1.0f + expf(-gte)) * up; }
// exp(x) = 2^(x log2 e): the statistics sum one hardware exp2 per logit
constexpr float kLog2e = 1.4426950408889634f;

struct TileK {
  const bf16_t* X;
  const bf16_t* W;
  void* Y;
  float* part;    // [segments][M][NG][Nout] fp32 partials (tiles split over workgroups only)
  int* counters;  // [grid][kCounterStride] arrival counters (idem), zero between launches
  int M, Nout, K, tiles_m, tiles_n;
  int part_bytes;
  float* stats;   // kEpiStore, nullable: [M][nch][2] (max, sum of exp) of each row over this tile's columns, entry tn
  int nch;
  int xkb, ykb;   // x (SwiGLU: y) stored k-blocked, [K/32][M][32]
  int grid;       // workgroups (launch only; the kernel reads gridDim)
  int par;        // one-segment split plans: every workgroup of a tile reduces a slice of its rows
  int par_l2;     // par, and partials may go through one XCD's L2 (see the split hand-off)
  unsigned foreign;  // segments that act as if dispatched elsewhere (tests of the fallback; normally 0)
  // RMSNorm folded into the neighbours (nullable).  Consumer: every output row
  // m is scaled by 1 / sqrt(sum_t ssq_in[m][t] / K + eps) (x was stored as
  // bf16(h * gain)).  Producer (kEpiResidual, slice-reduced splits only): with
  // h = y + x . w^T also xg = bf16(h * gain) (k-blocked [N/32][M][32] when
  // xg_kb) and ssq_out[m][t] = sum of h^2 over columns 128t .. 128t+127.
  const float* ssq_in;
  int nt_in;
  float eps;
  const bf16_t* gain;
  bf16_t* xg;
  float* ssq_out;
  int xg_kb, nt_out;
};

typedef __attribute__((address_space(3))) void lds_void;
constexpr int kMaxSsq4 = 16;  // folded-norm consumer: up to 64 sums-of-squares partials per row


// Split partials of a tile cut into nseg segments: [segment][M][NG][Nout]
// fp32, segment = position in k order.  The tile's rows are cut into nslice
// slices (rs = ceil(BM / nslice) rows each); slice sl, rows [m0 + sl * rs,
// m0 + (sl+1) * rs), is summed over all segments in k order, four columns per
// unit, and the epilogue applied to it.  Segment c's partial is read from
// this XCD's L2 when bit c of l2seg is set, else from memory.
template <int BM, int BN, int NG, int EPI>
__device__ void slice_reduce(const TileK& a, __amdgpu_buffer_rsrc_t prs, int nseg, unsigned l2seg, int nslice, int sl,
                             int m0, int n0, const float* s_rinv) {
  constexpr int NC = NG == 1 ? BN : BN / 2;  // output columns of the tile (per group)
  constexpr int C4 = NC / 4;
  static_assert(EPI != kEpiResidual || C4 % 32 == 0, "a row's 128-column segments are whole half-waves of units");
  const int M = a.M, Nout = a.Nout;
  const int rs = (BM + nslice - 1) / nslice;
  const int r0 = m0 + sl * rs, r1 = min(min(m0 + (sl + 1) * rs, m0 + BM), M);
  const int units = max(0, r1 - r0) * C4;
  auto poff = [&](int c, int m, int q, int n) { return (uint32_t)((((size_t)c * M + m) * NG + q) * Nout + n) * 4u; };
  // whole passes of the workgroup (every lane takes part in the norm
  // epilogue's butterfly), units past the slice or the matrix idle
  for (int u0 = 0; u0 < units; u0 += blockDim.x) {
    const int u = u0 + (int)threadIdx.x;
    const int m = r0 + min(u, units - 1) / C4, n = n0 + (u % C4) * 4;
    const bool ok = u < units && n < Nout;
    float part = 0.f;
    if (ok) {
    auto ld = [&](int c, int q) {
      return (l2seg >> c) & 1u ? xcd_load(prs, poff(c, m, q, n)) : coherent_load(prs, poff(c, m, q, n));
    };
    f32x4 v[NG];
#pragma unroll
    for (int q = 0; q < NG; ++q) v[q] = ld(0, q);
    // the other segments, four loads in flight per group at a time, added in k order
    for (int c0 = 1; c0 < nseg; c0 += 4) {
      f32x4 t[4][NG];
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int q = 0; q < NG; ++q) t[j][q] = ld(min(c0 + j, nseg - 1), q);
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if (c0 + j < nseg)
#pragma unroll
          for (int q = 0; q < NG; ++q) v[q] = v[q] + t[j][q];
    }
    if (a.ssq_in) {
      const float sc = s_rinv[m - m0];
#pragma unroll
      for (int q = 0; q < NG; ++q) v[q] *= sc;
    }
    if constexpr (EPI == kEpiStore) {
      *reinterpret_cast<f32x4*>(static_cast<float*>(a.Y) + (size_t)m * Nout + n) = v[0];
    } else if constexpr (EPI == kEpiResidual) {
      f32x4* p = reinterpret_cast<f32x4*>(static_cast<float*>(a.Y) + (size_t)m * Nout + n);
      const f32x4 hv = *p + v[0];
      *p = hv;
      if (a.xg) {  // the next RMSNorm's inputs
        const u32x2 gw = *reinterpret_cast<const u32x2*>(a.gain + n);
        u32x2 o;
        o[0] = pack_bf16x2(hv[0] * bf2f((bf16_t)(gw[0] & 0xffffu)), hv[1] * bf2f((bf16_t)(gw[0] >> 16)));
        o[1] = pack_bf16x2(hv[2] * bf2f((bf16_t)(gw[1] & 0xffffu)), hv[3] * bf2f((bf16_t)(gw[1] >> 16)));
        bf16_t* xp = a.xg_kb ? a.xg + ((size_t)(n >> 5) * M + m) * 32 + (n & 31) : a.xg + (size_t)m * Nout + n;
        *reinterpret_cast<u32x2*>(xp) = o;
        part = hv[0] * hv[0];
        part = fmaf(hv[1], hv[1], part);
        part = fmaf(hv[2], hv[2], part);
        part = fmaf(hv[3], hv[3], part);
      }
    } else {
      const f32x4 gt = v[0], up = v[NG - 1];
      u32x2 o;
      o[0] = pack_bf16x2(silu_mul(gt[0], up[0]), silu_mul(gt[1], up[1]));
      o[1] = pack_bf16x2(silu_mul(gt[2], up[2]), silu_mul(gt[3], up[3]));
      bf16_t* yp = a.ykb ? static_cast<bf16_t*>(a.Y) + ((size_t)(n >> 5) * M + m) * 32 + (n & 31)
                         : static_cast<bf16_t*>(a.Y) + (size_t)m * Nout + n;
      *reinterpret_cast<u32x2*>(yp) = o;
    }
    }
    if constexpr (EPI == kEpiResidual) {
      if (a.xg) {  // sum of h^2 over each 128-column segment: lane order, then a 5-step butterfly over its 32 units
        part += __shfl_xor(part, 1);
        part += __shfl_xor(part, 2);
        part += __shfl_xor(part, 4);
        part += __shfl_xor(part, 8);
        part += __shfl_xor(part, 16);
        if (u < units && (u % 32) == 0 && n < Nout) a.ssq_out[(size_t)m * a.nt_out + n / 128] = part;
      }
    }
  }
}

// SK: the stream-K loop over several segments per workgroup; without it a
// workgroup runs exactly one segment (the host launches such shapes only on
// grids whose shares never cross a tile boundary), which keeps the segment
// state out of the register budget of the 256 x 256 tiles.
template <int BM, int BN, int WM, int WN, int NBUF, int NG, int EPI, bool SK>
__global__ __launch_bounds__(WM * WN * 64) void gemm_tile_kernel(TileK a) {
  constexpr int NW = WM * WN;
  constexpr int TM = BM / WM / 16;                 // x fragments per wave
  constexpr int TN = BN / WN / 16;                 // weight fragments per wave
  constexpr int XU = BM / 16, WU = BN / 16;        // 1 KB units per stage
  // units each wave loads per stage; when they do not split evenly, the
  // surplus slots of the last waves load the stage's last unit again, to the
  // same LDS address (the same bytes), so every wave issues the same number
  // of loads and the load-counter waits below stay exact
  constexpr int UPW = (XU + WU + NW - 1) / NW;
  constexpr int STAGE = (XU + WU) * 512;           // bf16 elements per stage buffer
  constexpr int DIST = NBUF - 1;                   // stages in flight ahead of the one multiplied
  constexpr int HALF = BN / 2;                     // SwiGLU: gate rows, then up rows
  static_assert(NG == 1 || (TN % 2 == 0), "SwiGLU waves hold gate and up fragments in pairs");
  static_assert(DIST * UPW <= 63, "load counter range");
  __shared__ __attribute__((aligned(16))) bf16_t lds[NBUF * STAGE];
  __shared__ int s_last;
  __shared__ float s_rinv[BM];  // consumer of a folded RMSNorm: 1/rms of the tile's rows

  // Stream-K schedule over weight-tile columns.  The work of one M tile is
  // tiles_n x KU units (a unit: one output tile, 64 of k; units k-major
  // inside a weight tile).  Workgroup w = s tiles_m + tm takes M tile tm and
  // share s of the G' = G / tiles_m shares: units [s U' / G', (s+1) U' / G')
  // of the U' = tiles_n KU, so every workgroup gets the same amount of work
  // whatever the tile count, and the tiles_m workgroups of a share walk the
  // same weights at the same k (read once from HBM, then from L2).  A tile
  // covered by more than one share is a run of segments in k order; each
  // writes its partial and the last to arrive adds them in that order (fixed,
  // so the result does not depend on timing).  With G' = tiles_n x c for c
  // dividing KU this is a plain c-way split of K; with c = 1, one tile per
  // workgroup.
  // XCD-aware order: workgroup b runs on XCD b % 8; XCD x takes the x-th
  // contiguous run of w, so the M tiles of a share run on one XCD.
  const unsigned G = gridDim.x, bid = blockIdx.x;
  const unsigned gper = G >> 3, grem = G & 7, xcd = bid & 7, loc = bid >> 3;
  const unsigned w = xcd < grem ? xcd * (gper + 1) + loc : grem * (gper + 1) + (xcd - grem) * gper + loc;
  const int tm = __builtin_amdgcn_readfirstlane(w % a.tiles_m);
  const unsigned sh = w / a.tiles_m, GS = G / a.tiles_m;
  // The host keeps U' < 2^31 and G < 2^20.  The first unit of share v is
  // floor(v U' / G') = v q + floor(v r / G'), and the owner of unit X, the
  // largest v with floor(v U' / G') <= X, is floor(((X+1) G' - 1) / U') (in
  // fp64, exact below 2^53; the quotient is never within 1/U' of an integer it
  // is not).
  const unsigned KU = a.K / 64, U = (unsigned)a.tiles_n * KU;
  const unsigned uq = U / GS, ur = U % GS;
  auto first_unit = [&](unsigned v) { return v * uq + (unsigned)((unsigned long long)v * ur / GS); };
  auto owner = [&](unsigned X) { return (unsigned)((((double)X + 1.0) * GS - 1.0) / U); };
  unsigned unit = first_unit(sh);
  const unsigned unit_end = first_unit(sh + 1);

  const int M = a.M, Nout = a.Nout, K = a.K;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int r = lane & 15, g = lane >> 4;
  const int KS = K / 32, nto = Nout / 16;
  const int wv = __builtin_amdgcn_readfirstlane(wave);

  for (int seg = 0; unit < unit_end; ++seg) {
  // the segment's values are uniform: readfirstlane keeps them in scalar
  // registers across the main loop
  const int tn = __builtin_amdgcn_readfirstlane(unit / KU);
  const int ku0 = __builtin_amdgcn_readfirstlane(unit - tn * KU);
  const int ku1 = __builtin_amdgcn_readfirstlane(min(KU, ku0 + (unit_end - unit)));
  unit += ku1 - ku0;
  const int s_first = __builtin_amdgcn_readfirstlane(owner(tn * KU));
  const int nseg = __builtin_amdgcn_readfirstlane(owner(tn * KU + KU - 1)) - s_first + 1;
  const int slot = (int)sh - s_first;  // this segment's place in the tile's k order
  const int w_first = s_first * a.tiles_m + tm;  // owns the tile's counter
  if (seg > 0) __syncthreads();  // the previous tile's epilogue is done with LDS
  const int m0 = tm * BM;
  const int n0 = tn * (NG == 1 ? BN : HALF);

  // The units this wave loads: u = min(wave * UPW + q, XU + WU - 1); u < XU is x row tile u
  // (rows clamped into range: rows past the end are computed and never
  // stored), else weight tile u - XU (SwiGLU: gate tiles, then up tiles;
  // tiles past the edge clamped to the last one).  Address of stage st: the
  // uniform base ubase[q] + st * ustep[q] bytes plus the lane's 32-bit
  // offset vofs[q].
  const char* ubase[UPW];
  uint32_t ustep[UPW], vofs[UPW];
#pragma unroll
  for (int q = 0; q < UPW; ++q) {
    const int u = min(wv * UPW + q, XU + WU - 1);
    if (u < XU) {
      // row-major x: 64 bytes of each of 16 rows; k-blocked x: one 1 KB run
      const uint32_t row = (uint32_t)min(m0 + u * 16 + r, M - 1);
      ubase[q] = reinterpret_cast<const char*>(a.X);
      ustep[q] = a.xkb ? (uint32_t)M * 64u : 64u;
      vofs[q] = a.xkb ? (row * 32u + g * 8) * 2u : (row * (uint32_t)K + g * 8) * 2u;
    } else {
      const int t16 = u - XU;
      int T;
      if constexpr (NG == 1) T = min(n0 / 16 + t16, nto - 1);
      else T = t16 < HALF / 16 ? min(n0 / 16 + t16, nto - 1) : nto + min(n0 / 16 + t16 - HALF / 16, nto - 1);
      ubase[q] = reinterpret_cast<const char*>(a.W + ((size_t)(T >> 3) * KS * 8 + (T & 7)) * 512);
      ustep[q] = 8192;
      vofs[q] = lane * 16;
    }
  }
  // Unit q of stage st into buffer buf.  Written as assembly so that the
  // compiler, which cannot tell the stage buffers apart, does not wait for
  // these loads before every LDS read; the waits are explicit below.
  const uint32_t lds_base = (uint32_t)(uintptr_t)(lds_void*)lds;
  auto issue1 = [&](int q, int st, int buf) {
    const char* sb = ubase[q] + (size_t)st * ustep[q];
    const uint32_t dst = lds_base + (uint32_t)(buf * STAGE + min(wv * UPW + q, XU + WU - 1) * 512) * 2u;
    asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(vofs[q]), "s"(sb), "s"(dst)
                 : "memory", "m0");
  };
  auto issue = [&](int st, int buf) {
#pragma unroll
    for (int q = 0; q < UPW; ++q) issue1(q, st, buf);
  };
  // LDS unit of weight fragment j of this wave: wave base + a constant
  const int wub = XU + wn * (NG == 1 ? TN : TN / 2), xub = wm * TM;
  auto wofs = [](int j) { return NG == 1 ? j : (j < TN / 2 ? j : WU / 2 + j - TN / 2); };

  f32x4 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  // Per-buffer fragment read addresses, fixed for the whole loop: every read
  // below is one of these plus a compile-time offset (a ds_read immediate),
  // so the loop computes no LDS addresses.
  const bf16_t* wrd[NBUF];
  const bf16_t* xrd[NBUF];
#pragma unroll
  for (int b = 0; b < NBUF; ++b) {
    wrd[b] = lds + b * STAGE + wub * 512 + lane * 8;
    xrd[b] = lds + b * STAGE + xub * 512 + lane * 8;
  }
  auto ld16 = [](const bf16_t* p) { return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(p)); };

  // Fragments go through two register sets: those of stage st+1 are read
  // from LDS while stage st is multiplied.
  bf16x8 xf[2][TM], wf[2][TN];

  // a unit is two stages here (a stage is one 32-wide k-step)
  const int st0 = 2 * ku0, st1 = min(KS, 2 * ku1);
  // Prologue: stages st0 .. st0+NBUF-1 in flight, stage st0 read.  Stages
  // past the chunk re-load its last stage into a buffer nobody reads, so
  // every iteration issues the same number of loads and the wait counts
  // below are exact.
  // Folded-norm consumer: this thread's row of sums-of-squares partials
  // (thread t: row m0 + t), loaded ahead of the stages as assembly so that
  // the compiler adds no wait of its own (which would also drain the stages);
  // the prologue's wait below leaves only stage loads outstanding, so these
  // have landed by then.
  f32x4 ssq_v[kMaxSsq4];
  const bool rinv_row = a.ssq_in && seg == 0 && (int)threadIdx.x < BM;
  if (rinv_row) {
    const float* sp = a.ssq_in + (size_t)min(m0 + (int)threadIdx.x, M - 1) * a.nt_in;
#pragma unroll
    for (int q = 0; q < kMaxSsq4; ++q)
      if (q * 4 < a.nt_in) asm volatile("global_load_dwordx4 %0, %1, off" : "=v"(ssq_v[q]) : "v"(sp + 4 * q) : "memory");
  }
#pragma unroll
  for (int d = 0; d < NBUF; ++d) issue(min(st0 + d, st1 - 1), d);
  asm volatile("s_waitcnt vmcnt(%0)\n\ts_barrier" ::"n"((NBUF - 1) * UPW) : "memory");
  if (rinv_row) {  // 1/rms of row m0 + t (partials summed in order); read after later barriers
#pragma unroll
    for (int q = 0; q < kMaxSsq4; ++q) asm volatile("" : "+v"(ssq_v[q]));
    float sum = 0.f;
#pragma unroll
    for (int q = 0; q < kMaxSsq4; ++q)
      if (q * 4 < a.nt_in)
#pragma unroll
        for (int e = 0; e < 4; ++e) sum += ssq_v[q][e];
    s_rinv[threadIdx.x] = 1.0f / sqrtf(sum / (float)K + a.eps);
  }
#pragma unroll
  for (int j = 0; j < TN; ++j) wf[0][j] = ld16(wrd[0] + wofs(j) * 512);
#pragma unroll
  for (int i = 0; i < TM; ++i) xf[0][i] = ld16(xrd[0] + i * 512);
  // Step st (stage st sits in buffer (st - st0) % NBUF): stage st+1 has
  // landed in this wave's units once at most the NBUF-2 later stages' loads
  // are outstanding, and in every wave's after the barrier -- by which time
  // every wave's reads of stage st (issued during step st-1, completed before
  // the barrier) are done, so its buffer takes stage st+NBUF.  Then stage
  // st+1 is read while stage st is multiplied.
  // Each MFMA row i (TN multiplies) is preceded by this stage's share of the
  // loads for stage st+NBUF and of the fragment reads for stage st+1, so the
  // wave never stops issuing MFMAs for long (one wave per SIMD in the
  // 4-wave shape hides nothing behind another wave).
  constexpr int NRD = TM + TN;
  auto step = [&](auto pc, auto bc, int st) {
    constexpr int P = decltype(pc)::value, Q = 1 - P;
    constexpr int BUF = decltype(bc)::value, RBUF = (BUF + 1) % NBUF;
    const int nst = min(st + NBUF, st1 - 1);
    // LDS reads first, as a wait the compiler sees (so it knows every
    // fragment register has landed), then the loads and the barrier
    __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0)
    asm volatile("s_waitcnt vmcnt(%0)\n\ts_barrier" ::"n"((NBUF - 2) * UPW) : "memory");
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int q = i * UPW / TM; q < (i + 1) * UPW / TM; ++q) issue1(q, nst, BUF);
#pragma unroll
      for (int e = i * NRD / TM; e < (i + 1) * NRD / TM; ++e) {
        if (e < TN) wf[Q][e] = ld16(wrd[RBUF] + wofs(e) * 512);
        else xf[Q][e - TN] = ld16(xrd[RBUF] + (e - TN) * 512);
      }
#pragma unroll
      for (int j = 0; j < TN; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf[P][j], xf[P][i], acc[i][j], 0, 0, 0);
    }
    __builtin_amdgcn_sched_barrier(0);
  };
  // Unrolled so that the buffer and the register set of every step are
  // compile-time constants.
  constexpr int UNR = NBUF % 2 == 0 ? NBUF : 2 * NBUF;
  for (int st = st0; st < st1; st += UNR) {
    [&]<int... S>(std::integer_sequence<int, S...>) {
      ((st + S < st1 ? (step(std::integral_constant<int, S % 2>{}, std::integral_constant<int, S % NBUF>{}, st + S), 0) : 0), ...);
    }(std::make_integer_sequence<int, UNR>{});
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // the surplus loads, before LDS is reused or the workgroup exits

  // output coordinates of fragment (i, j): row m(i), columns n(j)..n(j)+3 of group q(j)
  auto out_m = [&](int i) { return m0 + wm * (BM / WM) + i * 16 + r; };
  auto out_n = [&](int j) {
    if constexpr (NG == 1) return n0 + wn * (BN / WN) + j * 16 + 4 * g;
    else return n0 + wn * (HALF / WN) + (j % (TN / 2)) * 16 + 4 * g;
  };
  auto out_q = [&](int j) { return NG == 1 ? 0 : j / (TN / 2); };

  if (nseg > 1) {
    // A split tile: publish the partial with device-coherent stores, count
    // arrivals, and let the last workgroup of the tile add the partials in k
    // order.  The counter of a split tile is that of its first workgroup
    // (no two split tiles share one).
    // With par_l2, a tile whose segments the XCD-aware order above puts in
    // one XCD's run exchanges its partials through that XCD's L2 (xcd_store /
    // xcd_load); a segment that did not land on the XCD round-robin dispatch
    // gives it ("foreign") writes through to memory and says so with its
    // arrival (bit 16 + slot of the counter), so that its partial is read from
    // memory and, when the tile's segments are mixed, one segment that is on
    // the expected XCD reduces the whole tile.  The sums are the same in every
    // case.
    const __amdgpu_buffer_rsrc_t prs = coherent_rsrc(a.part, a.part_bytes);
    auto poff = [&](int c, int m, int j) {
      return (uint32_t)((((size_t)c * M + m) * NG + out_q(j)) * Nout + out_n(j)) * 4u;
    };
    auto xcd_of = [&](unsigned v) {  // the XCD whose run holds logical workgroup v
      return v < grem * (gper + 1) ? v / (gper + 1) : grem + (v - grem * (gper + 1)) / max(gper, 1u);
    };
    const bool tile_l2 = a.par_l2 && !SK &&
                         xcd_of((unsigned)w_first) == xcd_of((unsigned)((s_first + nseg - 1) * a.tiles_m + tm));
    const bool foreign = tile_l2 && (xcd_id() != xcd || ((a.foreign >> slot) & 1u));
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const int m = out_m(i);
      if (m >= M) continue;
#pragma unroll
      for (int j = 0; j < TN; ++j)
        if (out_n(j) < Nout) {
          if (tile_l2 && !foreign) xcd_store(prs, poff(slot, m, j), acc[i][j]);
          else coherent_store(prs, poff(slot, m, j), acc[i][j]);
        }
    }
    __asm__ volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    int* cnt = a.counters + (size_t)w_first * kCounterStride;
    if constexpr (!SK) {
      if (a.par) {
        // Every workgroup of the tile waits for the tile's nseg partials,
        // then reduces its own slice of the tile's rows (the same k order
        // as the last-arriver reduction, so the same bits): nseg CUs share
        // the reduction instead of one reading all partials.  The host
        // launches this only on grids of at most one workgroup per CU, so
        // all of them are resident; the wait is still bounded, and a
        // timeout is flagged in the workspace's error word, which sits
        // right before the counter region.
        if (threadIdx.x == 0) {
          __hip_atomic_fetch_add(cnt, 1 + (foreign ? 1 << (16 + slot) : 0), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          int v = 0;
          for (int it = 0; ((v = __hip_atomic_load(cnt, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) & 0xffff) < nseg; ++it) {
            if (it >= kSplitSpinMax) {
              atomicOr(a.counters - kSplitErrOffset, kErrSplitWait);
              break;
            }
            __builtin_amdgcn_s_sleep(2);
          }
          s_last = (int)((unsigned)v >> 16);  // the foreign segments
        }
        __syncthreads();
        const unsigned fmask = (unsigned)s_last, all = (1u << nseg) - 1u;
        const unsigned l2seg = tile_l2 ? ~fmask & all : 0u;
        if (fmask != 0 && fmask != all) {
          // mixed: the first segment on the expected XCD reduces the whole tile
          if (slot == __builtin_ctz(l2seg)) slice_reduce<BM, BN, NG, EPI>(a, prs, nseg, l2seg, 1, 0, m0, n0, s_rinv);
        } else {
          slice_reduce<BM, BN, NG, EPI>(a, prs, nseg, l2seg, nseg, slot, m0, n0, s_rinv);
        }
        __asm__ volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();
        // the last to leave resets both counters for the next launch
        if (threadIdx.x == 0 &&
            __hip_atomic_fetch_add(cnt + 1, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == nseg - 1) {
          __hip_atomic_store(cnt, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          __hip_atomic_store(cnt + 1, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        return;
      }
    }
    if (threadIdx.x == 0)
      s_last = (__hip_atomic_fetch_add(cnt, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == nseg - 1);
    __syncthreads();
    if (!s_last) {
      if constexpr (SK) continue;
      else return;
    }
    if (threadIdx.x == 0) __hip_atomic_store(cnt, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);  // next launch
    // Sum all partials (this workgroup's own included, read back) in k
    // order; half of the row fragments at a time (rows [h TM / 2, (h+1) TM / 2),
    // which covers an odd TM too) keeps 16 loads in flight.
    // Fragments past the edge read a clamped in-range address and are dropped.
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      for (int c = 0; c < nseg; ++c) {
#pragma unroll
        for (int i = h * TM / 2; i < (h + 1) * TM / 2; ++i) {
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

  if (a.ssq_in) {
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const float sc = s_rinv[min(out_m(i), M - 1) - m0];
#pragma unroll
      for (int j = 0; j < TN; ++j) acc[i][j] *= sc;
    }
  }

  if constexpr (EPI == kEpiStore) {
    if (a.stats) {
      // Softmax statistics of each row over the tile's BN columns: a wave's
      // row (i, r) spans its TN fragments in the 4 lanes r + 16 g (max, then
      // the sum of exp (as 2^((v - max) log2 e)) in lane order and a 2-step butterfly -- a + b == b + a,
      // so the 4 lanes agree), then the WN waves of a row block merge in wave
      // order through LDS (the stage buffers are free).
      float* sst = reinterpret_cast<float*>(lds);  // [WM][WN][BM / WM][2]
      __syncthreads();
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        float mx = -INFINITY;
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (out_n(j) + e < Nout) mx = fmaxf(mx, acc[i][j][e]);
        mx = fmaxf(mx, __shfl_xor(mx, 16));
        mx = fmaxf(mx, __shfl_xor(mx, 32));
        float sum = 0.f;
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (out_n(j) + e < Nout) sum += __builtin_amdgcn_exp2f((acc[i][j][e] - mx) * kLog2e);
        sum += __shfl_xor(sum, 16);
        sum += __shfl_xor(sum, 32);
        if (g == 0) {
          const int rr = i * 16 + r;
          sst[((wm * WN + wn) * (BM / WM) + rr) * 2] = mx;
          sst[((wm * WN + wn) * (BM / WM) + rr) * 2 + 1] = sum;
        }
      }
      __syncthreads();
      for (int row = threadIdx.x; row < BM; row += NW * 64) {
        const int bm = row / (BM / WM), rr = row % (BM / WM), mrow = m0 + row;
        if (mrow >= M) continue;
        float m = -INFINITY, sum = 0.f;
        for (int w = 0; w < WN; ++w) {
          const float m2 = sst[((bm * WN + w) * (BM / WM) + rr) * 2], s2 = sst[((bm * WN + w) * (BM / WM) + rr) * 2 + 1];
          if (m2 == -INFINITY) continue;
          if (m == -INFINITY) {
            m = m2;
            sum = s2;
          } else if (m2 > m) {
            sum = sum * expf(m - m2) + s2;
            m = m2;
          } else {
            sum += s2 * expf(m2 - m);
          }
        }
        *reinterpret_cast<float2*>(a.stats + ((size_t)mrow * a.nch + tn) * 2) = float2{m, sum};
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
        bf16_t* yp = a.ykb ? static_cast<bf16_t*>(a.Y) + ((size_t)(n >> 5) * M + m) * 32 + (n & 31)
                           : static_cast<bf16_t*>(a.Y) + (size_t)m * Nout + n;
        *reinterpret_cast<u32x2*>(yp) = o;
      }
    }
  }
  if constexpr (!SK) break;
  }  // segments
}

template <int BM, int BN, int WM, int WN, int NBUF, bool SK>
hipError_t launch_shape(const TileK& a, int epi, hipStream_t s) {
  const dim3 grid(a.grid), block(WM * WN * 64);
  if (epi == kEpiStore) hipLaunchKernelGGL((gemm_tile_kernel<BM, BN, WM, WN, NBUF, 1, kEpiStore, SK>), grid, block, 0, s, a);
  else if (epi == kEpiResidual)
    hipLaunchKernelGGL((gemm_tile_kernel<BM, BN, WM, WN, NBUF, 1, kEpiResidual, SK>), grid, block, 0, s, a);
  else hipLaunchKernelGGL((gemm_tile_kernel<BM, BN, WM, WN, NBUF, 2, kEpiSwiglu, SK>), grid, block, 0, s, a);
  return hipGetLastError();
}
template <int BM, int BN, int WM, int WN, int NBUF>
hipError_t launch_shape_any(const TileK& a, int epi, bool one_segment, hipStream_t s) {
  return one_segment ? launch_shape<BM, BN, WM, WN, NBUF, false>(a, epi, s)
                     : launch_shape<BM, BN, WM, WN, NBUF, true>(a, epi, s);
}

}  // namespace

bool tile_one_segment(const GemmPlan& p, int K) {
  const long tiles = (long)p.ntiles * p.mblocks;
  return p.grid % tiles == 0 && p.grid / tiles <= K / 64;
}

int tile_bm(int cfg) {
  switch (cfg) {
    case kTile256x256: return 256;
    case kTile192x256: return 192;
    case kTile160x256: return 160;
    case kTile96x256:
    case kTile96x128: return 96;
    default: return 128;
  }
}
int tile_bn(int cfg) { return cfg == kTile128x128 || cfg == kTile96x128 ? 128 : 256; }

hipError_t launch_gemm_tile(const void* x, const void* w, void* y, int M, int N, int K, int epi, const GemmPlan& p,
                            int* counters, float* part, hipStream_t s, float* stats, bool x_kblocked,
                            bool y_kblocked, const GemmNorm* nm) {
  const int Nout = (epi == kEpiSwiglu) ? N / 2 : N;
  const bool split = p.part_bytes > 0;
  const long units = (long)p.ntiles * (K / 64);  // per M tile
  if (p.grid < p.mblocks || p.grid % p.mblocks || p.grid / p.mblocks > units || p.grid >= (1 << 20) ||
      units >= (1L << 31) || (split && (!part || !counters)))
    return hipErrorInvalidValue;
  TileK a{static_cast<const bf16_t*>(x), static_cast<const bf16_t*>(w), y, split ? part : nullptr,
          split ? counters : nullptr, M, Nout, K, p.mblocks, p.ntiles,
          (int)p.part_bytes, epi == kEpiStore ? stats : nullptr, (Nout + kStatChunk - 1) / kStatChunk,
          x_kblocked ? 1 : 0, y_kblocked ? 1 : 0, p.grid, 0, 0, 0u,
          nullptr, 0, 0.f, nullptr, nullptr, nullptr, 0, 0};
  const bool one_segment = tile_one_segment(p, K);
  a.par = split && one_segment && p.par && !a.stats && p.grid <= device_cus() ? 1 : 0;
  a.par_l2 = a.par && p.grid / ((long)p.ntiles * p.mblocks) <= kSplitL2MaxChunks ? 1 : 0;
  a.foreign = split_foreign_mask();
  if (nm) {
    if (nm->ssq_in) {
      // whole 16-byte loads of a row's partials
      if (nm->nt_in < 1 || nm->nt_in > 4 * kMaxSsq4 || nm->nt_in % 4) return hipErrorInvalidValue;
      a.ssq_in = nm->ssq_in, a.nt_in = nm->nt_in, a.eps = nm->eps;
    }
    if (nm->xg) {
      // the producer side lives in the slice reduction: residual plans whose
      // split tiles are reduced by all their workgroups
      if (epi != kEpiResidual || !a.par || !nm->gain || !nm->ssq_out || Nout % 32) return hipErrorInvalidValue;
      a.gain = static_cast<const bf16_t*>(nm->gain), a.xg = static_cast<bf16_t*>(nm->xg), a.ssq_out = nm->ssq_out;
      a.xg_kb = nm->xg_kb, a.nt_out = (Nout + 127) / 128;
    }
  }
  switch (p.tile) {
    // 8 waves of 128 x 64 (two per SIMD: one issues MFMAs while the other
    // waits on LDS or a barrier); one segment per workgroup only (the
    // stream-K loop's state does not fit beside the accumulators)
    case kTile256x256:
      if (!one_segment) return hipErrorInvalidValue;
      return launch_shape<256, 256, 2, 4, 4, false>(a, epi, s);
    // 8 waves of 96 x 64: windows of 3 x 128 (or 6 x 64) rows without a padded tile
    case kTile192x256: return launch_shape_any<192, 256, 2, 4, 4>(a, epi, one_segment, s);
    // 8 waves of 80 x 64: windows of 2 x 160 rows (320 = B 64 x (k+1) 5)
    case kTile160x256: return launch_shape_any<160, 256, 2, 4, 4>(a, epi, one_segment, s);
    // 8 waves of 48 x 64 and of 48 x 32: more, smaller tiles where the
    // weight matrix has few rows
    case kTile96x256: return launch_shape_any<96, 256, 2, 4, 4>(a, epi, one_segment, s);
    case kTile96x128: return launch_shape_any<96, 128, 2, 4, 4>(a, epi, one_segment, s);
    case kTile128x256: return launch_shape_any<128, 256, 2, 4, 4>(a, epi, one_segment, s);
    default: return launch_shape_any<128, 128, 2, 2, 4>(a, epi, one_segment, s);
  }
}

}  // namespace nj
