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
// ([D][16]), which makes that an 8-byte load.  K and V blocks are read
// straight into MFMA operand registers (64 contiguous bytes per lane for K).
// Softmax is online in the log2 domain; blocks are dealt round-robin to the 4
// waves, merged through LDS, and, when the grid splits the KV range, written
// as partials that a combine kernel merges in split order.
#include "common.h"
#include "kernels.h"

namespace nj {
namespace {

constexpr int kD = 128;  // head dim of the bf16 path
constexpr int kTargetWorkgroups = 512;

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
  bf16_t* out;
  int* err;
  int max_blocks, num_blocks, T, H, Hkv, bps;
  float scale_log2;
};

template <int RT>
__global__ __launch_bounds__(256) void attn_bf16_kernel(AttnK a) {
  const int pair = blockIdx.x, split = blockIdx.y, nsplit = gridDim.y;
  const int b = pair / a.Hkv, kvh = pair % a.Hkv;
  const int G = a.H / a.Hkv, R = a.T * G;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r16 = lane & 15, g = lane >> 4;

  int ctx = a.ctx[b];
  if (ctx < 0 || ctx + a.T > a.max_blocks * kBlock) {
    if (threadIdx.x == 0 && split == 0) flag_error(a.err, kErrContext);
    ctx = max(0, min(ctx, a.max_blocks * kBlock - a.T));
  }
  const int nb_ctx = (ctx + kBlock - 1) / kBlock;
  const int c0 = split * a.bps, c1 = min(c0 + a.bps, nb_ctx);
  const int ncached = max(0, c1 - c0);
  const int nent = ncached + (split == 0 ? 1 : 0);  // split 0 also takes the window block

  bf16x8 qf[RT][4];
  int qpos[RT];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    const int qc = min(rt * 16 + r16, R - 1);  // padding rows repeat the last real row
    const int i = qc / G, hh = qc % G;
    const bf16_t* src = a.q + ((size_t)(b * a.T + i) * a.H + kvh * G + hh) * kD + 32 * g;
#pragma unroll
    for (int s = 0; s < 4; ++s) qf[rt][s] = ld8(src + 8 * s);
    qpos[rt] = i;
  }

  float m_run[RT], l_run[RT];
  f32x4 o[RT][8];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    m_run[rt] = -INFINITY;
    l_run[rt] = 0.f;
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) o[rt][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  for (int e = wave; e < nent; e += 4) {
    const bool win = (e == ncached);
    const bf16_t* kb;
    const bf16_t* vb;
    int nvalid;
    if (!win) {
      const int j = c0 + e;
      const int phys = a.table[(size_t)b * a.max_blocks + j];
      if (phys < 0 || phys >= a.num_blocks) {
        if (lane == 0) flag_error(a.err, kErrBlock);
        continue;
      }
      kb = a.kp + ((size_t)phys * a.Hkv + kvh) * (kBlock * kD);
      vb = a.vp + ((size_t)phys * a.Hkv + kvh) * (kBlock * kD);
      nvalid = min(kBlock, ctx - j * kBlock);
    } else {
      kb = a.wk + ((size_t)b * a.Hkv + kvh) * (kBlock * kD);
      vb = a.wv + ((size_t)b * a.Hkv + kvh) * (kBlock * kD);
      nvalid = a.T;
    }
    bf16x8 kf[4];
    const bf16_t* krow = kb + r16 * kD + 32 * g;
#pragma unroll
    for (int s = 0; s < 4; ++s) kf[s] = ld8(krow + 8 * s);
    u32x2 vf[8];
#pragma unroll
    for (int dt = 0; dt < 8; ++dt)
      vf[dt] = *reinterpret_cast<const u32x2*>(vb + (16 * dt + r16) * kBlock + 4 * g);
    if (4 * g + 3 >= nvalid) {  // tokens past the valid ones may hold anything: zero them
      const int keep = nvalid - 4 * g;  // tokens of this lane kept: 0..3
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) {
        uint32_t lo = vf[dt][0], hi = vf[dt][1];
        if (keep <= 0) lo = 0u;
        else if (keep == 1) lo &= 0xffffu;
        if (keep <= 2) hi = 0u;
        else if (keep == 3) hi &= 0xffffu;
        vf[dt][0] = lo;
        vf[dt][1] = hi;
      }
    }
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      f32x4 st = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < 4; ++s) st = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[s], qf[rt][s], st, 0, 0, 0);
      float sc[4];
      float bm = -INFINITY;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int tok = 4 * g + i;
        const bool ok = tok < nvalid && (!win || tok <= qpos[rt]);
        sc[i] = ok ? st[i] * a.scale_log2 : -INFINITY;
        bm = fmaxf(bm, sc[i]);
      }
      bm = fmaxf(bm, __shfl_xor(bm, 16));
      bm = fmaxf(bm, __shfl_xor(bm, 32));
      const float mn = fmaxf(m_run[rt], bm);
      const float alpha = (mn == -INFINITY) ? 1.f : exp2f(m_run[rt] - mn);
      float p[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) p[i] = (sc[i] == -INFINITY) ? 0.f : exp2f(sc[i] - mn);
      l_run[rt] = l_run[rt] * alpha + ((p[0] + p[1]) + (p[2] + p[3]));
      m_run[rt] = mn;
      u32x2 pp;
      pp[0] = pack_bf16x2(p[0], p[1]);
      pp[1] = pack_bf16x2(p[2], p[3]);
      const bf16x4 pf = __builtin_bit_cast(bf16x4, pp);
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) {
        o[rt][dt] *= alpha;
        o[rt][dt] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(bf16x4, vf[dt]), pf, o[rt][dt],
                                                              0, 0, 0);
      }
    }
  }

  // merge the 4 waves, one 16-row tile at a time
  __shared__ float s_o[4][kD][17];
  __shared__ float s_m[4][16], s_l[4][16];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    float lsum = l_run[rt];
    lsum += __shfl_xor(lsum, 16);
    lsum += __shfl_xor(lsum, 32);
#pragma unroll
    for (int dt = 0; dt < 8; ++dt)
#pragma unroll
      for (int i = 0; i < 4; ++i) s_o[wave][16 * dt + 4 * g + i][r16] = o[rt][dt][i];
    if (g == 0) {
      s_m[wave][r16] = m_run[rt];
      s_l[wave][r16] = lsum;
    }
    __syncthreads();
    for (int idx = threadIdx.x; idx < 16 * kD; idx += 256) {
      const int qr16 = idx / kD, d = idx % kD;
      const int qr = rt * 16 + qr16;
      float mx = -INFINITY;
#pragma unroll
      for (int w = 0; w < 4; ++w) mx = fmaxf(mx, s_m[w][qr16]);
      float acc = 0.f, wsum = 0.f;
      if (mx != -INFINITY) {
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          const float f = (s_m[w][qr16] == -INFINITY) ? 0.f : exp2f(s_m[w][qr16] - mx);
          wsum += f * s_l[w][qr16];
          acc += f * s_o[w][d][qr16];
        }
      }
      if (qr < R) {
        if (nsplit == 1) {
          const int i = qr / G, hh = qr % G;
          a.out[((size_t)(b * a.T + i) * a.H + kvh * G + hh) * kD + d] = f2bf(acc / wsum);
        } else {
          const size_t base = ((size_t)pair * nsplit + split) * (RT * 16) + qr;
          a.part_o[base * kD + d] = acc;
          if (d == 0) {
            a.part_ml[base * 2] = mx;
            a.part_ml[base * 2 + 1] = wsum;
          }
        }
      }
    }
    __syncthreads();
  }
}

// Merge KV-split partials in split order: out = sum_s 2^(m_s - M) o_s / sum_s 2^(m_s - M) l_s.
// One workgroup per (sequence, KV head, query row), one thread per head dim.
__global__ __launch_bounds__(kD) void attn_combine_kernel(const float* __restrict__ part_o,
                                                          const float* __restrict__ part_ml,
                                                          bf16_t* __restrict__ out, int nsplit, int rpad, int T,
                                                          int H, int Hkv) {
  const int pair = blockIdx.x, qr = blockIdx.y, d = threadIdx.x;
  const int b = pair / Hkv, kvh = pair % Hkv, G = H / Hkv;
  float mx = -INFINITY;
  for (int s = 0; s < nsplit; ++s) mx = fmaxf(mx, part_ml[(((size_t)pair * nsplit + s) * rpad + qr) * 2]);
  float acc = 0.f, wsum = 0.f;
  for (int s = 0; s < nsplit; ++s) {
    const size_t base = ((size_t)pair * nsplit + s) * rpad + qr;
    const float m = part_ml[base * 2];
    const float f = (m == -INFINITY) ? 0.f : exp2f(m - mx);
    wsum += f * part_ml[base * 2 + 1];
    acc += f * part_o[base * kD + d];
  }
  const int i = qr / G, hh = qr % G;
  out[((size_t)(b * T + i) * H + kvh * G + hh) * kD + d] = f2bf(acc / wsum);
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

void attention_plan(int B, int Hkv, int T, int G, int max_blocks, int* nsplit, int* blocks_per_split) {
  (void)T;
  (void)G;
  const int pairs = B * Hkv;
  int ns = (kTargetWorkgroups + pairs - 1) / pairs;
  const int cap = (max_blocks + 7) / 8;  // at least ~8 cached blocks (2 per wave) per split
  if (ns > cap) ns = cap;
  if (ns < 1) ns = 1;
  int bps = (max_blocks + ns - 1) / ns;
  ns = (max_blocks + bps - 1) / bps;
  if (ns < 1) ns = 1;
  *nsplit = ns;
  *blocks_per_split = bps < 1 ? 1 : bps;
}

size_t attention_partial_floats(int B, int Hkv, int T, int G, int D) {
  const int rpad = ((T * G + 15) / 16) * 16;
  return (size_t)(B * Hkv + kTargetWorkgroups) * rpad * (D + 2);
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
          static_cast<const bf16_t*>(x.win_v), x.block_table, x.ctx, x.part_o, x.part_ml,
          static_cast<bf16_t*>(x.out), x.err, x.max_blocks, x.num_blocks, x.T, x.H, x.Hkv, x.blocks_per_split,
          (float)(1.4426950408889634 / sqrt((double)kD))};
  dim3 grid(x.B * x.Hkv, x.nsplit);
  switch (RT) {
    case 1: hipLaunchKernelGGL(attn_bf16_kernel<1>, grid, dim3(256), 0, s, a); break;
    case 2: hipLaunchKernelGGL(attn_bf16_kernel<2>, grid, dim3(256), 0, s, a); break;
    case 3: hipLaunchKernelGGL(attn_bf16_kernel<3>, grid, dim3(256), 0, s, a); break;
    default: hipLaunchKernelGGL(attn_bf16_kernel<4>, grid, dim3(256), 0, s, a); break;
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || x.nsplit == 1) return e;
  hipLaunchKernelGGL(attn_combine_kernel, dim3(x.B * x.Hkv, R), dim3(kD), 0, s, x.part_o, x.part_ml,
                     static_cast<bf16_t*>(x.out), x.nsplit, RT * 16, x.T, x.H, x.Hkv);
  return hipGetLastError();
}

}  // namespace nj
