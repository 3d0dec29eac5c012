// Paged verify attention: each sequence's k+1 window queries attend to its
// cached tokens (reached through the block table, 16 tokens per block) and
// causally to the window itself.
//
// bf16 path.  One workgroup (4 waves) per (sequence, KV head, KV split).  The
// G query heads sharing a KV head and the T = k+1 window positions are packed
// into R = T*G query rows (at most 64 = 4 tiles of 16), so every key and value
// byte read from HBM serves all of them.  Per 16-token block a wave computes
//   S^T (16 tokens x 16 rows) = K . Q^T      with 4 x mfma 16x16x32 bf16
// which leaves lane l holding tokens 4*(l>>4)+i of query row l&15 -- exactly
// the B operand of
//   O^T (16 dims x 16 rows) += V^T . P^T     with mfma 16x16x16 bf16,
// so the softmax numerators go straight from the score registers into the
// second product with no data exchange.  The A operand V^T needs 4
// consecutive tokens of one dim: V pages are stored dim-major inside a block
// ([D][16]), which makes that an 8-byte read.  Softmax is online in the log2
// domain.  When the grid splits the KV range, each split writes its partial
// (o, max, sum) and the last split to arrive merges them in split order.
#include <algorithm>
#include <climits>

#include "attn_work.h"
#include "common.h"
#include "kernels.h"

namespace nj {
namespace {

constexpr int kD = 128;  // head dim of the bf16 path
#ifndef NJ_ATTN_BUF
#define NJ_ATTN_BUF 2
#endif
#ifndef NJ_ATTN_CHUNK
#define NJ_ATTN_CHUNK 4
#endif
constexpr int kAttnBuf = NJ_ATTN_BUF;      // chunk buffers per workgroup (kAttnBuf - 1 chunks in flight)
constexpr int kAttnChunk = NJ_ATTN_CHUNK;  // cached blocks per chunk
// workgroups per CU that the chunk buffers leave room for (160 KB of LDS)
constexpr int attn_wgs_per_cu(int nbuf, int cb) { return (160 * 1024 - 1024) / (nbuf * cb * 8 * 1024); }

__device__ __forceinline__ bf16x8 ld8(const bf16_t* p) {
  return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(p));
}

struct AttnK {
  const bf16_t* q;
  const bf16_t* kp;
  const bf16_t* vp;
  const bf16_t* wk;
  const bf16_t* wv;
  const int32_t* table;
  const int32_t* ctx;
  float* part_o;
  float* part_ml;
  int* counters;  // [B*Hkv][kCounterStride] split arrivals, zero on entry (cleared before each launch)
  const AttnWork* work;  // [gridDim.x] the work list (attn_work.h)
  bf16_t* out;
  int* err;
  int max_blocks, num_blocks, T, H, Hkv;
  float scale_log2;
  int part_o_bytes, part_ml_bytes;
  int okbM;  // nonzero: out stored k-blocked, [H*kD/32][okbM][32] (okbM = B*T rows)
};

// output row m = b*T + i, column c = head * kD + d (4 consecutive columns)
__device__ __forceinline__ u32x2* out_at(const AttnK& a, int m, int c) {
  return reinterpret_cast<u32x2*>(a.okbM ? a.out + ((size_t)(c >> 5) * a.okbM + m) * 32 + (c & 31)
                                         : a.out + (size_t)m * a.H * kD + c);
}

// The workgroup
// streams its KV range in chunks of kCB blocks, loaded straight into LDS
// while earlier ones are multiplied out of LDS (NBUF buffers, NBUF-1 chunks in
// flight).  Waves are split into
// RTW row tiles x (4 / RTW) token phases: a wave multiplies its row tile
// against every (4/RTW)-th block of the chunk, and the phases of a tile are
// merged at the end.  LDS rows are XOR-swizzled in 16-byte (K) and 8-byte (V)
// units so that the fragment reads of 16 consecutive rows hit distinct banks.
constexpr int kKPieces = kBlock * kD / 8;  // 16-byte pieces per K (or V) block: 256

__device__ __forceinline__ int k_lds(int tok, int chunk16) {  // element offset in a K block [16][128]
  return tok * kD + ((chunk16 ^ tok) & 15) * 8;
}
__device__ __forceinline__ int v_lds(int dim, int unit8) {  // element offset in a V block [128][16]
  return dim * kBlock + ((unit8 ^ (((dim >> 3) & 1) << 1)) & 3) * 4;
}

// A split has written its partial (o, max, sum) with device-coherent stores;
// count it in, and let the last split of the (sequence, KV head) to arrive
// merge all splits in split order:
//   out = sum_s 2^(m_s - M) o_s / sum_s 2^(m_s - M) l_s.
// The per-split (m, l) of every query row go to LDS first and each row's
// weights 2^(m_s - M) are formed once; then each thread merges 4 head dims of
// one query row per unit, with the loads of all splits of a unit in flight
// together.  `lds` is the kernel's staging buffer (free by now).
constexpr int kMergeSplits = 8;   // split partials loaded together per unit
constexpr int kMergeUnits = 4;    // units merged together per thread
__device__ void split_arrive(const AttnK& a, int pair, int nsplit, int slot0, int R, int RT, int G, int b, int kvh,
                             __amdgpu_buffer_rsrc_t ors, __amdgpu_buffer_rsrc_t mrs, float* lds, int lds_floats) {
  __shared__ int s_last;
  __asm__ volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  if (threadIdx.x == 0)
    s_last = (__hip_atomic_fetch_add(a.counters + pair * kCounterStride, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == nsplit - 1);
  __syncthreads();
  if (!s_last) return;
  const int rpad = RT * 16;
  const size_t pbase = (size_t)slot0 * rpad;
  // s_f[qr][sp]: weight 2^(m_sp - M) of split sp for row qr (0 for empty
  // splits); s_w[qr]: 1 / sum_sp weight * l_sp.  The (m, l) of every row and
  // split are loaded in one pass.
  float* s_f = lds;
  float* s_l = lds + R * nsplit;
  float* s_w = lds + 2 * R * nsplit;
  if (2 * R * nsplit + R <= lds_floats) {
    for (int u = threadIdx.x; u < R * nsplit; u += 256) {
      const int qr = u / nsplit, sp = u % nsplit;
      const uint32_t off = (uint32_t)(((pbase + (size_t)sp * rpad + qr) * 2) * 4);
      s_f[u] = coherent_load_f32(mrs, off);
      s_l[u] = coherent_load_f32(mrs, off + 4);
    }
    __syncthreads();
    for (int qr = threadIdx.x; qr < R; qr += 256) {
      float mx = -INFINITY;
      for (int sp = 0; sp < nsplit; ++sp) mx = fmaxf(mx, s_f[qr * nsplit + sp]);
      // an empty split wrote only its -inf marker: its l and o slots hold
      // whatever the workspace held before, so it is masked out, not weighted 0
      float wsum = 0.f;
      for (int sp = 0; sp < nsplit; ++sp) {
        const float m = s_f[qr * nsplit + sp];
        const float f = (m == -INFINITY) ? 0.f : exp2f(m - mx);
        s_f[qr * nsplit + sp] = f;
        if (m != -INFINITY) wsum += f * s_l[qr * nsplit + sp];
      }
      s_w[qr] = 1.0f / wsum;
    }
    __syncthreads();
    // each unit: 4 head dims of one row.  A thread takes up to kMergeUnits
    // units at a time and issues the loads of all their splits (kMergeSplits
    // at a time) together.
    const int nunits = R * (kD / 4);
    for (int ub = 0; ub < nunits; ub += 256 * kMergeUnits) {
      f32x4 acc[kMergeUnits];
#pragma unroll
      for (int q = 0; q < kMergeUnits; ++q) acc[q] = f32x4{0.f, 0.f, 0.f, 0.f};
      for (int s0 = 0; s0 < nsplit; s0 += kMergeSplits) {
        f32x4 ov[kMergeUnits][kMergeSplits];
#pragma unroll
        for (int q = 0; q < kMergeUnits; ++q) {
          const int u = min(ub + (int)threadIdx.x + q * 256, nunits - 1);
          const int qr = u / (kD / 4), d = (u % (kD / 4)) * 4;
#pragma unroll
          for (int j = 0; j < kMergeSplits; ++j) {
            const int sp = min(s0 + j, nsplit - 1);
            ov[q][j] = coherent_load(ors, (uint32_t)(((pbase + (size_t)sp * rpad + qr) * kD + d) * 4));
          }
        }
#pragma unroll
        for (int q = 0; q < kMergeUnits; ++q) {
          const int qr = min(ub + (int)threadIdx.x + q * 256, nunits - 1) / (kD / 4);
#pragma unroll
          for (int j = 0; j < kMergeSplits; ++j)
            if (s0 + j < nsplit && s_f[qr * nsplit + s0 + j] != 0.f) acc[q] += s_f[qr * nsplit + s0 + j] * ov[q][j];
        }
      }
#pragma unroll
      for (int q = 0; q < kMergeUnits; ++q) {
        const int u = ub + (int)threadIdx.x + q * 256;
        if (u >= nunits) break;
        const int qr = u / (kD / 4), d = (u % (kD / 4)) * 4;
        const float inv = s_w[qr];
        const int i = qr / G, hh = qr % G;
        u32x2 o;
        o[0] = pack_bf16x2(acc[q][0] * inv, acc[q][1] * inv);
        o[1] = pack_bf16x2(acc[q][2] * inv, acc[q][3] * inv);
        *out_at(a, b * a.T + i, (kvh * G + hh) * kD + d) = o;
      }
    }
    return;
  }
  // too many splits to stage (not reached by attention_plan's splits): direct loads
  for (int u = threadIdx.x; u < R * (kD / 4); u += 256) {
    const int qr = u / (kD / 4), d = (u % (kD / 4)) * 4;
    float mx = -INFINITY;
    for (int sp = 0; sp < nsplit; ++sp)
      mx = fmaxf(mx, coherent_load_f32(mrs, (uint32_t)(((pbase + (size_t)sp * rpad + qr) * 2) * 4)));
    f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
    float wsum = 0.f;
    for (int sp = 0; sp < nsplit; ++sp) {
      const size_t base = pbase + (size_t)sp * rpad + qr;
      const float m = coherent_load_f32(mrs, (uint32_t)((base * 2) * 4));
      if (m == -INFINITY) continue;  // empty split: only its marker was written
      const float f = exp2f(m - mx);
      wsum += f * coherent_load_f32(mrs, (uint32_t)((base * 2 + 1) * 4));
      acc += f * coherent_load(ors, (uint32_t)((base * kD + d) * 4));
    }
    const float inv = 1.0f / wsum;
    const int i = qr / G, hh = qr % G;
    u32x2 o;
    o[0] = pack_bf16x2(acc[0] * inv, acc[1] * inv);
    o[1] = pack_bf16x2(acc[2] * inv, acc[3] * inv);
    *out_at(a, b * a.T + i, (kvh * G + hh) * kD + d) = o;
  }
}

template <int RTW, int NBUF, int kCB>
__global__ __launch_bounds__(256, attn_wgs_per_cu(NBUF, kCB)) void attn_lds_kernel(AttnK a) {
  constexpr int NTP = 4 / RTW;  // token phases per row tile
  constexpr int KV_ELEMS = kCB * kBlock * kD;  // one chunk of K (or V)
  constexpr int WPB = 4 / kCB;  // waves loading one block (its K and V halves when 2)
  constexpr int UPW = 8 / WPB;  // 1 KB load instructions per wave and chunk
  static_assert(kCB == 2 || kCB == 4, "a chunk's blocks split evenly over the 4 waves");
  __shared__ __attribute__((aligned(16))) bf16_t smem[NBUF * 2 * KV_ELEMS];  // [buf][K|V][chunk], 32 KB per buffer
  const AttnWork item = a.work[blockIdx.x];
  if (item.nsplit == 0) return;  // the list is shorter than the grid
  const int b = item.b, kvh = item.kvh, split = item.split, nsplit = item.nsplit;
  const int pair = b * a.Hkv + kvh, slot0 = item.slot0;
  const int G = a.H / a.Hkv, R = a.T * G, RT = (R + 15) / 16;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r16 = lane & 15, g = lane >> 4;
  const int rt = wave % RTW, tp = wave / RTW;

  const int ctx = item.ctx >= 0 ? item.ctx : ~item.ctx;
  if (item.ctx < 0 && threadIdx.x == 0 && split == 0) flag_error(a.err, kErrContext);
  // this split's share of the cached blocks (shares differ by at most one
  // block); split 0 also takes the window block, as its first chunk: it is in
  // L2 (just written), so its compute overlaps the first cached chunk's loads
  const int c0 = item.c0, c1 = item.c1;
  const int ncc = (c1 - c0 + kCB - 1) / kCB;  // cached chunks
  const int wch = split == 0 ? 1 : 0;         // window chunks
  const int nchunks = ncc + wch;

  const __amdgpu_buffer_rsrc_t ors = coherent_rsrc(a.part_o, a.part_o_bytes);
  const __amdgpu_buffer_rsrc_t mrs = coherent_rsrc(a.part_ml, a.part_ml_bytes);
  if (nchunks == 0) {  // no blocks of this sequence for this split: mark its rows empty for the merge
    for (int qr = threadIdx.x; qr < R; qr += 256)
      coherent_store_f32(mrs, (uint32_t)(((((size_t)slot0 + split) * (RT * 16) + qr) * 2) * 4), -INFINITY);
    split_arrive(a, pair, nsplit, slot0, R, RT, G, b, kvh, ors, mrs, reinterpret_cast<float*>(smem),
                 (int)(sizeof(smem) / sizeof(float)));
    return;
  }
  bf16x8 qf[4];
  int qpos;
  float m_run = -INFINITY, l_run = 0.f;
  f32x4 o[8];
#pragma unroll
  for (int dt = 0; dt < 8; ++dt) o[dt] = f32x4{0.f, 0.f, 0.f, 0.f};

  // chunk ch: blocks [j0, j0 + nblk) of the cached range, or the window block
  auto chunk_blocks = [&](int ch, int& j0, int& nblk) {
    if (ch >= wch) {
      j0 = c0 + (ch - wch) * kCB;
      nblk = min(kCB, c1 - j0);
    } else {
      j0 = -1;
      nblk = 1;
    }
  };
  // Chunk loads go from memory straight into LDS (global_load_lds_dwordx4):
  // a block is 4 K and 4 V instructions of 1 KB, loaded by one wave (chunks
  // of 4 blocks) or by two (K and V; chunks of 2), and
  // lane i's 16 bytes land at byte 16 i of the instruction's KB -- so each lane
  // fetches the global piece that the swizzled layout keeps there.  NBUF
  // buffers, NBUF-1 chunks in flight.  A block's page id is read with a scalar
  // load one chunk before its pages; blocks past the chunk, or with a bad id,
  // load the window block (valid memory, never read as cache).  Every chunk
  // issues the same UPW loads per wave, so the wait counts below are exact.
  const int wv = __builtin_amdgcn_readfirstlane(wave);
  uint32_t kofs[4], vofs[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int tok = 4 * j + (lane >> 4), slot = lane & 15;
    kofs[j] = (uint32_t)(tok * kD + ((slot ^ tok) & 15) * 8) * 2u;
    const int dim = 32 * j + (lane >> 1), hv = (lane & 1) ^ ((dim >> 3) & 1);
    vofs[j] = (uint32_t)(dim * kBlock + hv * 8) * 2u;
  }
  const bf16_t* win_k = a.wk + ((size_t)b * a.Hkv + kvh) * (kBlock * kD);
  const bf16_t* win_v = a.wv + ((size_t)b * a.Hkv + kvh) * (kBlock * kD);
  const uint32_t lds0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) void*)smem;
  bool bad = false;
  // Page ids: lane l of wave w holds the id of block w of cached chunk
  // idbase + l, read 64 chunks at a time (a split longer than 64 chunks
  // reloads, waiting for its loads in flight); a chunk's id is then a lane
  // read, with no memory access in the loop.  kNoBlock (not a table value):
  // load the window block.  Any table entry outside [0, num_blocks) of a block
  // inside the context, -1 included, is a bad block.
  constexpr int kNoBlock = INT_MIN;
  int idv = kNoBlock, idbase = -64;
  auto block_id = [&](int ch) {
    if (ch < wch || ch >= nchunks) return kNoBlock;
    const int cc = ch - wch;
    if (cc - idbase >= 64) {
      idbase = cc;
      const int blk = c0 + (cc + lane) * kCB + wv / WPB;
      idv = (cc + lane < ncc && blk < c1) ? a.table[(size_t)b * a.max_blocks + blk] : kNoBlock;
      __builtin_amdgcn_s_waitcnt(0x0f70);  // vmcnt(0)
    }
    return __builtin_amdgcn_readlane(idv, cc - idbase);
  };
  auto issue = [&](int ch, int id) {
    const int buf = ch % NBUF;
    int ph = __builtin_amdgcn_readfirstlane(id);
    if (ph != kNoBlock && (ph < 0 || ph >= a.num_blocks)) {
      bad = true;
      ph = kNoBlock;
    }
    const size_t off = ((size_t)max(ph, 0) * a.Hkv + kvh) * (kBlock * kD);
    const bf16_t* kb = ph >= 0 ? a.kp + off : win_k;
    const bf16_t* vb = ph >= 0 ? a.vp + off : win_v;
    const uint32_t kd = lds0 + (uint32_t)(buf * 2 * KV_ELEMS + (wv / WPB) * kBlock * kD) * 2u;
    const uint32_t vd = kd + (uint32_t)KV_ELEMS * 2u;
    if (WPB == 1 || wv % 2 == 0) {
#pragma unroll
      for (int j = 0; j < 4; ++j)
        asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(kofs[j]), "s"(kb), "s"(kd + j * 1024)
                     : "memory", "m0");
    }
    if (WPB == 1 || wv % 2 == 1) {
#pragma unroll
      for (int j = 0; j < 4; ++j)
        asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(vofs[j]), "s"(vb), "s"(vd + j * 1024)
                     : "memory", "m0");
    }
  };
  for (int d = 0; d < NBUF - 1; ++d) issue(d, block_id(d));
  int ph_pre = block_id(NBUF - 1);
  // q after the prologue's chunks, and a wait the compiler sees: from here on
  // no load of its own is outstanding, so it adds no load waits in the loop
  // (which would also wait for the chunks in flight)
  {
    const int qc = min(rt * 16 + r16, R - 1);  // padding rows repeat the last real row
    const int i = qc / G, hh = qc % G;
    const bf16_t* src = a.q + ((size_t)(b * a.T + i) * a.H + kvh * G + hh) * kD + 32 * g;
#pragma unroll
    for (int s = 0; s < 4; ++s) qf[s] = ld8(src + 8 * s);
    qpos = i;
  }
  __builtin_amdgcn_s_waitcnt(0x0f70);  // vmcnt(0)
  for (int ch = 0; ch < nchunks; ++ch) {
    // this wave's loads of chunk ch have landed once at most the later
    // NBUF-2 chunks' are outstanding; after the barrier every wave's have, and
    // every wave is done with chunk ch-1, whose buffer takes chunk ch+NBUF-1
    asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"((NBUF - 2) * UPW) : "memory");
    issue(ch + NBUF - 1, ph_pre);
    ph_pre = block_id(ch + NBUF);
    int j0, nblk;
    chunk_blocks(ch, j0, nblk);
    const bool win = j0 < 0;
    const bf16_t* ks = smem + (ch % NBUF) * 2 * KV_ELEMS;
    const bf16_t* vs = ks + KV_ELEMS;
    if (rt < RT) {
      // Blocks bi and bi + NTP together: their score products are two
      // independent chains, and one cross-lane max, one exp2 of the running
      // max and one rescale of the accumulators serve both.
      for (int bi = tp; bi < nblk; bi += 2 * NTP) {
        const bool two = bi + NTP < nblk;  // uniform
        bf16x8 kf[2][4];
        u32x2 vf[2][8];
        int nvalid[2];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          if (h == 1 && !two) break;
          const int blk = bi + h * NTP;
          nvalid[h] = win ? a.T : min(kBlock, ctx - (j0 + blk) * kBlock);
          const bf16_t* kb = ks + blk * kBlock * kD;
          const bf16_t* vb = vs + blk * kBlock * kD;
#pragma unroll
          for (int s = 0; s < 4; ++s) kf[h][s] = ld8(kb + k_lds(r16, 4 * g + s));
#pragma unroll
          for (int dt = 0; dt < 8; ++dt) vf[h][dt] = *reinterpret_cast<const u32x2*>(vb + v_lds(16 * dt + r16, g));
          if (4 * g + 3 >= nvalid[h]) {  // tokens past the valid ones may hold anything: zero them
            const int keep = nvalid[h] - 4 * g;
#pragma unroll
            for (int dt = 0; dt < 8; ++dt) {
              uint32_t lo = vf[h][dt][0], hi = vf[h][dt][1];
              if (keep <= 0) lo = 0u;
              else if (keep == 1) lo &= 0xffffu;
              if (keep <= 2) hi = 0u;
              else if (keep == 3) hi &= 0xffffu;
              vf[h][dt][0] = lo;
              vf[h][dt][1] = hi;
            }
          }
        }
        f32x4 st[2] = {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}};
#pragma unroll
        for (int s = 0; s < 4; ++s) {
          st[0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[0][s], qf[s], st[0], 0, 0, 0);
          if (two) st[1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[1][s], qf[s], st[1], 0, 0, 0);
        }
        float sc[2][4];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
#pragma unroll
          for (int i = 0; i < 4; ++i) sc[h][i] = st[h][i] * a.scale_log2;
          if (h == 1 && !two) {
#pragma unroll
            for (int i = 0; i < 4; ++i) sc[h][i] = -INFINITY;
          } else if (win || nvalid[h] < kBlock) {  // uniform: only a partial or the window block masks tokens
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const int tok = 4 * g + i;
              if (!(tok < nvalid[h] && (!win || tok <= qpos))) sc[h][i] = -INFINITY;
            }
          }
        }
        float bm = fmaxf(fmaxf(fmaxf(sc[0][0], sc[0][1]), fmaxf(sc[0][2], sc[0][3])),
                         fmaxf(fmaxf(sc[1][0], sc[1][1]), fmaxf(sc[1][2], sc[1][3])));
        bm = fmaxf(bm, __shfl_xor(bm, 16));
        bm = fmaxf(bm, __shfl_xor(bm, 32));
        const float mn = fmaxf(m_run, bm);
        // exponents are <= 0 here: the hardware exp2 (v_exp_f32) gives
        // exp2(-inf) = 0 for masked tokens; a row with nothing valid yet
        // (mn = -inf) keeps p = 0
        const float ms = mn == -INFINITY ? 0.f : mn;
        const float alpha = __builtin_amdgcn_exp2f(m_run - ms);
        float p[2][4];
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
          for (int i = 0; i < 4; ++i) p[h][i] = __builtin_amdgcn_exp2f(sc[h][i] - ms);
        l_run = l_run * alpha + (((p[0][0] + p[0][1]) + (p[0][2] + p[0][3])) + ((p[1][0] + p[1][1]) + (p[1][2] + p[1][3])));
        m_run = mn;
        bf16x4 pf[2];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          u32x2 pp;
          pp[0] = pack_bf16x2(p[h][0], p[h][1]);
          pp[1] = pack_bf16x2(p[h][2], p[h][3]);
          pf[h] = __builtin_bit_cast(bf16x4, pp);
        }
        // the accumulators move only when some row's running max rose (uniform branch)
        if (__builtin_amdgcn_ballot_w64(alpha != 1.f)) {
#pragma unroll
          for (int dt = 0; dt < 8; ++dt) o[dt] *= alpha;
        }
#pragma unroll
        for (int dt = 0; dt < 8; ++dt) {
          o[dt] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(bf16x4, vf[0][dt]), pf[0], o[dt], 0, 0, 0);
          if (two)
            o[dt] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(bf16x4, vf[1][dt]), pf[1], o[dt], 0, 0, 0);
        }
      }
    }
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // the surplus loads, before LDS is reused
  __syncthreads();
  if (bad && lane == 0) flag_error(a.err, kErrBlock);  // bad is per wave

  // merge the token phases of each row tile (LDS reused), then store or write partials
  float* s_o = reinterpret_cast<float*>(smem);  // [NTP][kD][17]
  float* s_m = s_o + NTP * kD * 17;             // [NTP][16]
  float* s_l = s_m + NTP * 16;
  for (int t = 0; t < RT; ++t) {
    if (rt == t) {
      float lsum = l_run;
      lsum += __shfl_xor(lsum, 16);
      lsum += __shfl_xor(lsum, 32);
#pragma unroll
      for (int dt = 0; dt < 8; ++dt)
#pragma unroll
        for (int i = 0; i < 4; ++i) s_o[(tp * kD + 16 * dt + 4 * g + i) * 17 + r16] = o[dt][i];
      if (g == 0) {
        s_m[tp * 16 + r16] = m_run;
        s_l[tp * 16 + r16] = lsum;
      }
    }
    __syncthreads();
    // thread: 4 consecutive head dims of one query row per unit (2 units)
    for (int u = threadIdx.x; u < 16 * (kD / 4); u += 256) {
      const int qr16 = u / (kD / 4), d = (u % (kD / 4)) * 4;
      const int qr = t * 16 + qr16;
      float mx = -INFINITY;
#pragma unroll
      for (int w = 0; w < NTP; ++w) mx = fmaxf(mx, s_m[w * 16 + qr16]);
      f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
      float wsum = 0.f;
      if (mx != -INFINITY) {
#pragma unroll
        for (int w = 0; w < NTP; ++w) {
          const float f = (s_m[w * 16 + qr16] == -INFINITY) ? 0.f : exp2f(s_m[w * 16 + qr16] - mx);
          wsum += f * s_l[w * 16 + qr16];
#pragma unroll
          for (int e = 0; e < 4; ++e) acc[e] += f * s_o[(w * kD + d + e) * 17 + qr16];
        }
      }
      if (qr < R) {
        if (nsplit == 1) {
          const int i = qr / G, hh = qr % G;
          u32x2 ov;
          ov[0] = pack_bf16x2(acc[0] / wsum, acc[1] / wsum);
          ov[1] = pack_bf16x2(acc[2] / wsum, acc[3] / wsum);
          *out_at(a, b * a.T + i, (kvh * G + hh) * kD + d) = ov;
        } else {
          const size_t base = ((size_t)slot0 + split) * (RT * 16) + qr;
          coherent_store(ors, (uint32_t)((base * kD + d) * 4), acc);
          if (d == 0) {
            coherent_store_f32(mrs, (uint32_t)(base * 2 * 4), mx);
            coherent_store_f32(mrs, (uint32_t)((base * 2 + 1) * 4), wsum);
          }
        }
      }
    }
    __syncthreads();
  }
  if (nsplit > 1)
    split_arrive(a, pair, nsplit, slot0, R, RT, G, b, kvh, ors, mrs, reinterpret_cast<float*>(smem),
                 (int)(sizeof(smem) / sizeof(float)));
}

// fp32 path: one workgroup per (sequence, query head, window position); scores
// in LDS, exact softmax, then one thread per output dim.
struct AttnF {
  const float* q;
  const float* kp;
  const float* vp;
  const float* wk;
  const float* wv;
  const int32_t* table;
  const int32_t* ctx;
  float* out;
  int* err;
  int max_blocks, num_blocks, T, H, Hkv, D;
  float scale;
};

__global__ __launch_bounds__(128) void attn_f32_kernel(AttnF a) {
  extern __shared__ float sc[];
  __shared__ float red[2];
  __shared__ float wred[2];
  const int b = blockIdx.x / a.H, h = blockIdx.x % a.H, i = blockIdx.y;
  const int G = a.H / a.Hkv, kvh = h / G, D = a.D;
  int ctx = a.ctx[b];
  if (ctx < 0 || ctx + a.T > a.max_blocks * kBlock) {
    if (threadIdx.x == 0 && h == 0 && i == 0) flag_error(a.err, kErrContext);
    ctx = max(0, min(ctx, a.max_blocks * kBlock - a.T));
  }
  const int n = ctx + i + 1;
  const float* qr = a.q + ((size_t)(b * a.T + i) * a.H + h) * D;
  float mx = -INFINITY;
  for (int t = threadIdx.x; t < n; t += blockDim.x) {
    const float* kr;
    if (t < ctx) {
      const int phys = a.table[(size_t)b * a.max_blocks + t / kBlock];
      if (phys < 0 || phys >= a.num_blocks) {
        flag_error(a.err, kErrBlock);
        sc[t] = -INFINITY;
        continue;
      }
      kr = a.kp + (((size_t)phys * a.Hkv + kvh) * kBlock + t % kBlock) * D;
    } else {
      kr = a.wk + (((size_t)b * a.Hkv + kvh) * kBlock + (t - ctx)) * D;
    }
    float dot = 0.f;
    for (int d = 0; d < D; ++d) dot = fmaf(qr[d], kr[d], dot);
    sc[t] = dot * a.scale;
    mx = fmaxf(mx, sc[t]);
  }
  for (int o = 32; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o));
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = mx;
  __syncthreads();
  mx = fmaxf(red[0], red[1]);
  float sum = 0.f;
  for (int t = threadIdx.x; t < n; t += blockDim.x) {
    const float e = (sc[t] == -INFINITY) ? 0.f : expf(sc[t] - mx);
    sc[t] = e;
    sum += e;
  }
  for (int o = 32; o > 0; o >>= 1) sum += __shfl_xor(sum, o);
  if ((threadIdx.x & 63) == 0) wred[threadIdx.x >> 6] = sum;
  __syncthreads();
  sum = wred[0] + wred[1];
  for (int d = threadIdx.x; d < D; d += blockDim.x) {
    float acc = 0.f;
    for (int t = 0; t < n; ++t) {
      float v;
      if (t < ctx) {
        const int phys = a.table[(size_t)b * a.max_blocks + t / kBlock];
        if (phys < 0 || phys >= a.num_blocks) continue;
        v = a.vp[(((size_t)phys * a.Hkv + kvh) * D + d) * kBlock + t % kBlock];
      } else {
        v = a.wv[(((size_t)b * a.Hkv + kvh) * D + d) * kBlock + (t - ctx)];
      }
      acc = fmaf(sc[t], v, acc);
    }
    a.out[((size_t)(b * a.T + i) * a.H + h) * D + d] = acc / sum;
  }
}

}  // namespace

int attention_plan(int B, int Hkv, int max_blocks) {
  // Workgroups of the work list: one per (sequence, KV head) plus up to
  // kExtraWorkgroups more, and no more than the splits of kMinSplitBlocks
  // blocks the longest possible context could use.  The list sizes the
  // splits from the actual context lengths to fit this grid, so a long
  // sequence gets proportionally more splits than a short one.  Once the
  // pairs alone fill half of the resident attention workgroups, fewer extra
  // ones: the grid runs in rounds anyway, and longer splits pay their fixed
  // start-up and merge once per more blocks (measured: 8B B=64 k=4 and the
  // 7B shape at B=256 k=7 fastest with 128 extra, B=8 with 512).
  const int pairs = B * Hkv;
  const long cap = (long)pairs * std::max(1, (max_blocks + kMinSplitBlocks - 1) / kMinSplitBlocks);
  const int extra = 2 * pairs <= attn_wgs_per_cu(kAttnBuf, kAttnChunk) * device_cus() ? kExtraWorkgroups
                                                                                      : std::min(kExtraWorkgroups, kExtraWorkgroupsLarge);
  return (int)std::max<long>(pairs, std::min<long>((long)pairs + extra, cap));
}

bool attention_orders(int nwg) { return nwg > attn_wgs_per_cu(kAttnBuf, kAttnChunk) * device_cus(); }

size_t attention_work_bytes(int B, int Hkv) { return (size_t)(B * Hkv + kExtraWorkgroups) * sizeof(AttnWork); }

size_t attention_partial_floats(int B, int Hkv, int T, int G, int D) {
  const int rpad = ((T * G + 15) / 16) * 16;
  return (size_t)(B * Hkv + kExtraWorkgroups) * rpad * (D + 2);
}

namespace {
// One workgroup: the work list of the next attention launches, and (when
// counters is given) their split arrival counters cleared.
__global__ __launch_bounds__(256) void attn_plan_kernel(const int32_t* __restrict__ ctx, int B, int Hkv, int T,
                                                        int max_blocks, int nwg, int order, AttnWork* __restrict__ work,
                                                        int* __restrict__ counters) {
  __shared__ int scratch[attn_work_scratch_ints(256)];
  if (counters)
    for (int u = threadIdx.x; u < B * Hkv; u += 256) counters[u * kCounterStride] = 0;
  build_attn_work<256>(ctx, B, Hkv, T, max_blocks, nwg, order != 0, work, scratch);
}
}  // namespace

hipError_t launch_attn_plan(const int32_t* ctx, int B, int Hkv, int T, int max_blocks, int nwg, void* work,
                            int* counters, hipStream_t s) {
  if (nwg < B * Hkv || nwg > B * Hkv + kExtraWorkgroups) return hipErrorInvalidValue;
  hipLaunchKernelGGL(attn_plan_kernel, dim3(1), dim3(256), 0, s, ctx, B, Hkv, T, max_blocks, nwg,
                     attention_orders(nwg) ? 1 : 0, static_cast<AttnWork*>(work), counters);
  return hipGetLastError();
}

hipError_t launch_attention(const AttnArgs& x, hipStream_t s) {
  const int G = x.H / x.Hkv;
  if (x.dtype == kF32) {
    AttnF a{static_cast<const float*>(x.q), static_cast<const float*>(x.k_pages),
            static_cast<const float*>(x.v_pages), static_cast<const float*>(x.win_k),
            static_cast<const float*>(x.win_v), x.block_table, x.ctx, static_cast<float*>(x.out), x.err,
            x.max_blocks, x.num_blocks, x.T, x.H, x.Hkv, x.D, 1.0f / sqrtf((float)x.D)};
    const size_t lds = (size_t)x.max_blocks * kBlock * sizeof(float);
    hipLaunchKernelGGL(attn_f32_kernel, dim3(x.B * x.H, x.T), dim3(128), lds, s, a);
    return hipGetLastError();
  }
  const int R = x.T * G, RT = (R + 15) / 16;
  AttnK a{static_cast<const bf16_t*>(x.q), static_cast<const bf16_t*>(x.k_pages),
          static_cast<const bf16_t*>(x.v_pages), static_cast<const bf16_t*>(x.win_k),
          static_cast<const bf16_t*>(x.win_v), x.block_table, x.ctx, x.part_o, x.part_ml, x.counters,
          x.work, static_cast<bf16_t*>(x.out), x.err, x.max_blocks, x.num_blocks, x.T, x.H, x.Hkv,
          (float)(1.4426950408889634 / sqrt((double)kD)),
          (int)std::min<size_t>(attention_partial_floats(x.B, x.Hkv, x.T, G, kD) / (kD + 2) * kD * 4, INT32_MAX),
          (int)std::min<size_t>(attention_partial_floats(x.B, x.Hkv, x.T, G, kD) / (kD + 2) * 2 * 4, INT32_MAX),
          x.out_kblocked ? x.B * x.T : 0};
  if (!x.work || x.wgs < x.B * x.Hkv || x.wgs > x.B * x.Hkv + kExtraWorkgroups) return hipErrorInvalidValue;
  dim3 grid(x.wgs);
  switch (RT) {
    case 1: hipLaunchKernelGGL((attn_lds_kernel<1, kAttnBuf, kAttnChunk>), grid, dim3(256), 0, s, a); break;
    case 2: hipLaunchKernelGGL((attn_lds_kernel<2, kAttnBuf, kAttnChunk>), grid, dim3(256), 0, s, a); break;
    default: hipLaunchKernelGGL((attn_lds_kernel<4, kAttnBuf, kAttnChunk>), grid, dim3(256), 0, s, a); break;
  }
  return hipGetLastError();
}

}  // namespace nj
