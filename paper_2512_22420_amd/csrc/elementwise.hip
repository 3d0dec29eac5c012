// Small per-row kernels of the verify step: embedding gather fused with the
// first RMSNorm, RMSNorm, RoPE with the window K/V store, and the KV append
// of accepted rows.  All are HBM/latency bound and tiny next to the GEMMs.
#include "attn_work.h"
#include "common.h"
#include "kernels.h"

namespace nj {
namespace {

constexpr int kNormThreads = 256;
constexpr int kNormMaxPer = 8;  // float4 groups per thread: d <= 8192

__device__ __forceinline__ void load4(const float* p, float* v) {
  const f32x4 q = *reinterpret_cast<const f32x4*>(p);
  v[0] = q[0], v[1] = q[1], v[2] = q[2], v[3] = q[3];
}
__device__ __forceinline__ void load4(const bf16_t* p, float* v) {
  const u32x2 q = *reinterpret_cast<const u32x2*>(p);
  v[0] = __uint_as_float(q[0] << 16), v[1] = __uint_as_float(q[0] & 0xffff0000u);
  v[2] = __uint_as_float(q[1] << 16), v[3] = __uint_as_float(q[1] & 0xffff0000u);
}
__device__ __forceinline__ void store4(float* p, const float* v) {
  *reinterpret_cast<f32x4*>(p) = f32x4{v[0], v[1], v[2], v[3]};
}
__device__ __forceinline__ void store4(bf16_t* p, const float* v) {
  u32x2 q;
  q[0] = pack_bf16x2(v[0], v[1]);
  q[1] = pack_bf16x2(v[2], v[3]);
  *reinterpret_cast<u32x2*>(p) = q;
}

// x = h / sqrt(mean(h^2) + eps) * gain for one row held in registers
// (d % 4 == 0, d <= 4 * kNormThreads * kNormMaxPer).
template <typename T>
__device__ __forceinline__ void norm_row(const float (&hv)[kNormMaxPer][4], const T* __restrict__ gain,
                                         T* __restrict__ X, int row, int kbM, int d, float eps, float* sh) {
  float ss = 0.f;
#pragma unroll
  for (int it = 0; it < kNormMaxPer; ++it) {
    const int j = (it * kNormThreads + threadIdx.x) * 4;
    if (j < d)
#pragma unroll
      for (int e = 0; e < 4; ++e) ss = fmaf(hv[it][e], hv[it][e], ss);
  }
  ss = block_sum<kNormThreads>(ss, sh);
  const float r = 1.0f / sqrtf(ss / (float)d + eps);
#pragma unroll
  for (int it = 0; it < kNormMaxPer; ++it) {
    const int j = (it * kNormThreads + threadIdx.x) * 4;
    if (j < d) {
      float gv[4], o[4];
      load4(gain + j, gv);
#pragma unroll
      for (int e = 0; e < 4; ++e) o[e] = hv[it][e] * r * gv[e];
      // row-major [M][d], or k-blocked [d/32][M][32] for the LDS-tiled GEMM
      store4(kbM ? X + ((size_t)(j >> 5) * kbM + row) * 32 + (j & 31) : X + (size_t)row * d + j, o);
    }
  }
}

struct RopeFreqHead {  // theta^(-2j/128) for the 64 rotation pairs of a 128-dim head, from the host in fp64
  double inv_freq[64];
};

// Row `row` (window position i of sequence b) of the step's RoPE table:
// rope_cs[row][j] = (cos, sin) of (ctx_b + i) * theta^(-2j/128), the angle in
// fp64 with the range reduction done against 2 pi in two parts, the sincos in
// fp32 on the reduced argument.  Threads 0..63 of the workgroup.
// c: the sequence's context length (already loaded); run by threads 0..63.
__device__ __forceinline__ void rope_table_row(int c, const RopeFreqHead& f, int row, int i,
                                               float* __restrict__ rope_cs) {
  if (threadIdx.x < 64) {
    const int j = threadIdx.x;
    const double ang = (double)(max(c, 0) + i) * f.inv_freq[j];
    const double kq = rint(ang * 0.15915494309189535);
    const double red = fma(-kq, 6.283185307179586, ang) - kq * 2.4492935982947064e-16;
    float sn, cs;
    sincosf((float)red, &sn, &cs);
    rope_cs[((size_t)row * 64 + j) * 2] = cs;
    rope_cs[((size_t)row * 64 + j) * 2 + 1] = sn;
  }
}

template <typename T>
__global__ __launch_bounds__(kNormThreads) void embed_norm_kernel(
    const int32_t* __restrict__ last, const int32_t* __restrict__ drafts, int T_, const T* __restrict__ embed,
    const T* __restrict__ gain, float* __restrict__ h, T* __restrict__ x, int d, int V, float eps,
    int* __restrict__ err, int kbM, AttnPlan plan, const int32_t* __restrict__ ctx, RopeFreqHead f,
    float* __restrict__ rope_cs) {
  __shared__ float sh[kNormThreads / kWave];
  // the extra workgroup (dispatched first, so it overlaps the rows): the
  // attention's work list
  if (plan.work && blockIdx.x == 0) {
    __shared__ int scratch[attn_work_scratch_ints(kNormThreads)];
    build_attn_work<kNormThreads>(plan.ctx, plan.B, plan.Hkv, plan.T, plan.max_blocks, plan.nwg, plan.order != 0, plan.work,
                                  scratch);
    return;
  }
  const int row = blockIdx.x - (plan.work ? 1 : 0), b = row / T_, i = row % T_;
  // the token id and the context length load together; the RoPE math runs
  // while the embedding row is in flight
  int tok = (i == 0) ? last[b] : drafts[b * (T_ - 1) + i - 1];
  const int c = rope_cs && threadIdx.x < 64 ? ctx[b] : 0;
  if (tok < 0 || tok >= V) {
    if (threadIdx.x == 0) flag_error(err, kErrToken);
    tok = 0;
  }
  const T* e = embed + (size_t)tok * d;
  float* hr = h + (size_t)row * d;
  float hv[kNormMaxPer][4];
#pragma unroll
  for (int it = 0; it < kNormMaxPer; ++it) {
    const int j = (it * kNormThreads + threadIdx.x) * 4;
    if (j < d) load4(e + j, hv[it]);
  }
  if (rope_cs) rope_table_row(c, f, row, i, rope_cs);
#pragma unroll
  for (int it = 0; it < kNormMaxPer; ++it) {
    const int j = (it * kNormThreads + threadIdx.x) * 4;
    if (j < d) store4(hr + j, hv[it]);
  }
  norm_row<T>(hv, gain, x, row, kbM, d, eps, sh);
}

// bf16 path with the RMSNorm folded into the GEMMs: h = E[id], x = bf16(h *
// gain) and ssq[row][t] = sum of h^2 over columns 128t .. 128t+127 (the 32
// threads of a 128-column tile: lane order, then a 5-step butterfly), which
// the first GEMM turns into its row scale.
// It also writes the RoPE table of the step, rope_cs[row][j] = (cos, sin) of
// pos * theta^(-j/64), pos = ctx[b] + i, for the 64 rotation pairs of a
// 128-dim head (angle formed and reduced to [-pi, pi] in fp64, then fp32
// sin/cos, as in rope_window_kernel); every head and layer of the step uses it.

// With hin (fp32 [rows][d]) the rows are read from there instead of the
// embedding and h is not written: the same inputs for a given residual stream
// (the pre-attention stage entry point).
__global__ __launch_bounds__(kNormThreads) void embed_gather_kernel(
    const int32_t* __restrict__ last, const int32_t* __restrict__ drafts, int T_, const bf16_t* __restrict__ embed,
    const bf16_t* __restrict__ gain, float* __restrict__ h, bf16_t* __restrict__ x, float* __restrict__ ssq, int d,
    int V, int* __restrict__ err, const int32_t* __restrict__ ctx, RopeFreqHead f, float* __restrict__ rope_cs,
    const float* __restrict__ hin, AttnPlan plan) {
  // the extra workgroup (dispatched first, so it overlaps the rows): the
  // attention's work list
  if (plan.work && blockIdx.x == 0) {
    __shared__ int scratch[attn_work_scratch_ints(kNormThreads)];
    build_attn_work<kNormThreads>(plan.ctx, plan.B, plan.Hkv, plan.T, plan.max_blocks, plan.nwg, plan.order != 0, plan.work,
                                  scratch);
    return;
  }
  const int row = blockIdx.x - (plan.work ? 1 : 0), b = row / T_, i = row % T_;
  // Every load of the row goes out before any store: the token id and the
  // context length together, then the embedding (or residual) row and the
  // gains, under which the RoPE math runs.
  int tok = 0;
  if (!hin) tok = (i == 0) ? last[b] : drafts[b * (T_ - 1) + i - 1];
  const int c = rope_cs && threadIdx.x < 64 ? ctx[b] : 0;
  const float* src32 = hin ? hin + (size_t)row * d : nullptr;
  const bf16_t* e = nullptr;
  if (!hin) {
    if (tok < 0 || tok >= V) {
      if (threadIdx.x == 0) flag_error(err, kErrToken);
      tok = 0;
    }
    e = embed + (size_t)tok * d;
  }
  const int nt = (d + 127) / 128;
  float hv[kNormMaxPer][4], gv[kNormMaxPer][4];
#pragma unroll
  for (int it = 0; it < kNormMaxPer; ++it) {
    const int j = (it * kNormThreads + threadIdx.x) * 4;
#pragma unroll
    for (int q = 0; q < 4; ++q) hv[it][q] = gv[it][q] = 0.f;
    if (j < d) {
      if (hin) load4(src32 + j, hv[it]);
      else load4(e + j, hv[it]);
      load4(gain + j, gv[it]);
    }
  }
  if (rope_cs) rope_table_row(c, f, row, i, rope_cs);
#pragma unroll
  for (int it = 0; it < kNormMaxPer; ++it) {
    const int j = (it * kNormThreads + threadIdx.x) * 4;
    if (j >= ((d + 127) / 128) * 128) break;  // uniform per 32-lane tile
    float part = 0.f;
    if (j < d) {
      float o[4];
      if (!hin) store4(h + (size_t)row * d + j, hv[it]);
#pragma unroll
      for (int q = 0; q < 4; ++q) o[q] = hv[it][q] * gv[it][q];
      store4(x + (size_t)row * d + j, o);
      part = hv[it][0] * hv[it][0];
      part = fmaf(hv[it][1], hv[it][1], part);
      part = fmaf(hv[it][2], hv[it][2], part);
      part = fmaf(hv[it][3], hv[it][3], part);
    }
    part += __shfl_xor(part, 1);
    part += __shfl_xor(part, 2);
    part += __shfl_xor(part, 4);
    part += __shfl_xor(part, 8);
    part += __shfl_xor(part, 16);
    if ((threadIdx.x & 31) == 0) ssq[(size_t)row * nt + j / 128] = part;
  }
}

template <typename T>
__global__ __launch_bounds__(kNormThreads) void rmsnorm_kernel(const float* __restrict__ h,
                                                               const T* __restrict__ gain, T* __restrict__ x,
                                                               int d, float eps, int kbM) {
  __shared__ float sh[kNormThreads / kWave];
  const float* hr = h + (size_t)blockIdx.x * d;
  float hv[kNormMaxPer][4];
#pragma unroll
  for (int it = 0; it < kNormMaxPer; ++it) {
    const int j = (it * kNormThreads + threadIdx.x) * 4;
    if (j < d) load4(hr + j, hv[it]);
  }
  norm_row<T>(hv, gain, x, blockIdx.x, kbM, d, eps, sh);
}

// RoPE and the window K/V store.  One thread per rotation pair (j, j + D/2) of
// one head of one window row; workgroups cover (row, group of heads), so no
// thread walks a loop of dependent loads.  The pair turns by
// pos * theta^(-2j/D): theta^(-2j/D) comes from the host in fp64, the angle is
// formed and reduced to [-pi, pi] in fp64 (positions reach thousands of
// radians), then an fp32 sin/cos of the small argument.  q goes to
// q_out[row][h][:], k to win_k[b][g][i][:], v to win_v[b][g][:][i]; workgroups of
// row i == 0 also zero the unused slots T..15 of the window blocks so that
// masked lanes never read stale data.
template <typename T>
__global__ __launch_bounds__(256) void rope_window_kernel(const float* __restrict__ qkv,
                                                          const int32_t* __restrict__ ctx, int T_, int H,
                                                          int Hkv, int D, RopeFreq f, T* __restrict__ q_out,
                                                          T* __restrict__ win_k, T* __restrict__ win_v,
                                                          int32_t* __restrict__ ctx_snap, int* __restrict__ attn_cnt) {
  const int half = D / 2;
  const int hpb = blockDim.x / half;  // heads per workgroup
  const int row = blockIdx.x, b = row / T_, i = row % T_;
  const int hd = blockIdx.y * hpb + threadIdx.x / half, j = threadIdx.x % half;
  // the positions this step uses, for the KV append that follows it
  if (ctx_snap && i == 0 && blockIdx.y == 0 && threadIdx.x == 0) ctx_snap[b] = ctx[b];
  // the split counters of the attention launch that follows start at zero
  if (attn_cnt && i == 0 && blockIdx.y == 0)
    for (int g = threadIdx.x; g < Hkv; g += blockDim.x) attn_cnt[(b * Hkv + g) * kCounterStride] = 0;
  if (hd >= H + 2 * Hkv) return;
  const float* src = qkv + (size_t)row * (H + 2 * Hkv) * D + (size_t)hd * D;
  if (hd < H + Hkv) {
    const double ang = (double)(max(ctx[b], 0) + i) * f.inv_freq[j];
    const double kq = rint(ang * 0.15915494309189535);
    const double red = fma(-kq, 6.283185307179586, ang) - kq * 2.4492935982947064e-16;
    float sn, cs;
    sincosf((float)red, &sn, &cs);
    const float a = src[j], bb = src[j + half];
    const float ra = a * cs - bb * sn, rb = bb * cs + a * sn;
    T* dst;
    if (hd < H) {
      dst = q_out + ((size_t)row * H + hd) * D;
    } else {
      const int g = hd - H;
      dst = win_k + (((size_t)b * Hkv + g) * kBlock + i) * D;
      if (i == 0)
        for (int slot = T_; slot < kBlock; ++slot) {
          T* z = win_k + (((size_t)b * Hkv + g) * kBlock + slot) * D;
          z[j] = from_f<T>(0.f);
          z[j + half] = from_f<T>(0.f);
        }
    }
    dst[j] = from_f<T>(ra);
    dst[j + half] = from_f<T>(rb);
  } else {
    const int g = hd - H - Hkv;
    T* vb = win_v + ((size_t)b * Hkv + g) * D * kBlock;
    vb[(size_t)j * kBlock + i] = from_f<T>(src[j]);
    vb[(size_t)(j + half) * kBlock + i] = from_f<T>(src[j + half]);
    if (i == 0)
      for (int slot = T_; slot < kBlock; ++slot) {
        vb[(size_t)j * kBlock + slot] = from_f<T>(0.f);
        vb[(size_t)(j + half) * kBlock + slot] = from_f<T>(0.f);
      }
  }
}

constexpr int kMaxAppendLayers = 64;
struct PagePtrs {
  void* k[kMaxAppendLayers];
  void* v[kMaxAppendLayers];
};

// KV append.  grid (pieces, B, layers of this launch): one thread per (window
// row j, KV head g, 16-byte group of head dims) of one sequence and layer; rows
// past n_b exit at once.  K is copied as one 16-byte vector (the page row is
// contiguous), V element by element (pages keep V dim-major inside a block).
// Positions come from the context lengths the verify step read (its RoPE
// positions); the last launch also moves context_lens[b] past the new rows.
template <typename T>
__global__ __launch_bounds__(256) void kv_append_kernel(PagePtrs pages, int layer0, int last_launch,
                                                        const T* __restrict__ win_k, const T* __restrict__ win_v,
                                                        const int32_t* __restrict__ table, int max_blocks,
                                                        int num_blocks, const int32_t* __restrict__ ctx_snap,
                                                        int32_t* __restrict__ ctx, const int32_t* __restrict__ acc,
                                                        int B, int k, int Hkv, int D, int* __restrict__ err) {
  constexpr int EV = 16 / sizeof(T);  // elements per 16-byte group
  const int b = blockIdx.y, lc = blockIdx.z, l = layer0 + lc;
  const int groups = D / EV, u = blockIdx.x * blockDim.x + threadIdx.x;
  if (u >= (k + 1) * Hkv * groups) return;
  const int j = u / (Hkv * groups), rem = u % (Hkv * groups), g = rem / groups, e0 = (rem % groups) * EV;
  // the window row's values do not depend on n or the position: their loads
  // go out together with those of n and the context length
  const size_t wb = ((size_t)l * B + b) * Hkv + g;
  const u32x4 kv = *reinterpret_cast<const u32x4*>(win_k + (wb * kBlock + j) * D + e0);
  const T* vs = win_v + (wb * D + e0) * kBlock + j;
  T vv[EV];
#pragma unroll
  for (int e = 0; e < EV; ++e) vv[e] = vs[(size_t)e * kBlock];
  const int n = acc[b], c = ctx_snap[b];
  const bool lead = u == 0 && lc == 0;
  if (n < 0 || n > k) {
    if (lead) flag_error(err, kErrAccept);
    return;
  }
  if (c < 0 || c + k + 1 > max_blocks * kBlock) {
    if (lead) flag_error(err, kErrContext);
    return;
  }
  if (u == 0 && last_launch) ctx[b] = c + n + 1;
  if (j > n) return;
  const int pos = c + j;
  const int phys = table[(size_t)b * max_blocks + pos / kBlock];
  if (phys < 0 || phys >= num_blocks) {
    flag_error(err, kErrBlock);
    return;
  }
  const int slot = pos % kBlock;
  T* kp = static_cast<T*>(pages.k[lc]);
  T* vp = static_cast<T*>(pages.v[lc]);
  *reinterpret_cast<u32x4*>(kp + (((size_t)phys * Hkv + g) * kBlock + slot) * D + e0) = kv;
  T* vd = vp + (((size_t)phys * Hkv + g) * D + e0) * kBlock + slot;
#pragma unroll
  for (int e = 0; e < EV; ++e) vd[(size_t)e * kBlock] = vv[e];
}

__global__ void fill_i32_kernel(int32_t* p, int32_t v, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

__global__ void copy_i32_kernel(int32_t* __restrict__ dst, const int32_t* __restrict__ src, int n, int stride) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) dst[i] = src[(size_t)i * stride];
}

// RoPE and the window K/V store for bf16 heads of 128 dims: one workgroup
// per (sequence, head) covers the window's T rows, so the window blocks are
// written whole (slots T..15 zero) with 8- and 16-byte stores.  Thread t:
// row t / 16, rotation pairs (j, j + 64) for j = 4 (t % 16) .. +3.  V goes
// through LDS to come out dim-major ([128][16], 32 bytes per dim).  Angles as
// in rope_window_kernel.
__global__ __launch_bounds__(256) void rope_window_d128_kernel(const float* __restrict__ qkv,
                                                               const int32_t* __restrict__ ctx, int T_, int H,
                                                               int Hkv, RopeFreq f, bf16_t* __restrict__ q_out,
                                                               bf16_t* __restrict__ win_k, bf16_t* __restrict__ win_v,
                                                               int32_t* __restrict__ ctx_snap,
                                                               int* __restrict__ attn_cnt) {
  __shared__ float sv[kBlock][132];
  const int b = blockIdx.x, hd = blockIdx.y, t = threadIdx.x;
  const int i = t >> 4, j0 = 4 * (t & 15);
  const int nh = H + 2 * Hkv;
  if (hd == 0) {
    // the positions this step uses, for the KV append that follows it; and
    // the split counters of the attention launch that follows start at zero
    if (ctx_snap && t == 0) ctx_snap[b] = ctx[b];
    if (attn_cnt && t < Hkv) attn_cnt[(b * Hkv + t) * kCounterStride] = 0;
  }
  const float* src = qkv + ((size_t)(b * T_ + min(i, T_ - 1)) * nh + hd) * 128;
  if (hd < H + Hkv) {
    float ro[4], rh[4];
    if (i < T_) {
      const f32x4 a = *reinterpret_cast<const f32x4*>(src + j0), c = *reinterpret_cast<const f32x4*>(src + 64 + j0);
      const double pos = (double)(max(ctx[b], 0) + i);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const double ang = pos * f.inv_freq[j0 + e];
        const double kq = rint(ang * 0.15915494309189535);
        const double red = fma(-kq, 6.283185307179586, ang) - kq * 2.4492935982947064e-16;
        float sn, cs;
        sincosf((float)red, &sn, &cs);
        ro[e] = a[e] * cs - c[e] * sn;
        rh[e] = c[e] * cs + a[e] * sn;
      }
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) ro[e] = rh[e] = 0.f;
    }
    bf16_t* dst;
    if (hd < H) {
      if (i >= T_) return;
      dst = q_out + ((size_t)(b * T_ + i) * H + hd) * 128;
    } else {
      dst = win_k + (((size_t)b * Hkv + (hd - H)) * kBlock + i) * 128;  // rows T..15 zero
    }
    u32x2 lo, hi;
    lo[0] = pack_bf16x2(ro[0], ro[1]);
    lo[1] = pack_bf16x2(ro[2], ro[3]);
    hi[0] = pack_bf16x2(rh[0], rh[1]);
    hi[1] = pack_bf16x2(rh[2], rh[3]);
    *reinterpret_cast<u32x2*>(dst + j0) = lo;
    *reinterpret_cast<u32x2*>(dst + 64 + j0) = hi;
  } else {
    const f32x4 z = f32x4{0.f, 0.f, 0.f, 0.f};
    const f32x4 a = i < T_ ? *reinterpret_cast<const f32x4*>(src + j0) : z;
    const f32x4 c = i < T_ ? *reinterpret_cast<const f32x4*>(src + 64 + j0) : z;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      sv[i][j0 + e] = a[e];
      sv[i][64 + j0 + e] = c[e];
    }
    __syncthreads();
    const int d = t >> 1, h8 = (t & 1) * 8;  // dim d, slots h8 .. h8+7
    u32x4 o;
#pragma unroll
    for (int e = 0; e < 4; ++e) o[e] = pack_bf16x2(sv[h8 + 2 * e][d], sv[h8 + 2 * e + 1][d]);
    bf16_t* vb = win_v + ((size_t)b * Hkv + (hd - H - Hkv)) * 128 * kBlock;
    *reinterpret_cast<u32x4*>(vb + d * kBlock + h8) = o;
  }
}

}  // namespace

hipError_t launch_embed_norm(int dtype, const int32_t* last, const int32_t* drafts, int B, int T, const void* embed,
                             const void* gain, float* h, void* x, int d, int V, float eps, int* err,
                             hipStream_t s, bool x_kblocked, const AttnPlan* plan, const int32_t* ctx, float theta,
                             float* rope_cs) {
  const int kbM = x_kblocked ? B * T : 0;
  const AttnPlan pl = plan ? *plan : AttnPlan{};
  RopeFreqHead f{};
  if (rope_cs)
    for (int j = 0; j < 64; ++j) f.inv_freq[j] = pow((double)theta, -2.0 * j / 128);
  const dim3 grid(B * T + (pl.work ? 1 : 0));
  if (dtype == kF32)
    hipLaunchKernelGGL(embed_norm_kernel<float>, grid, dim3(kNormThreads), 0, s, last, drafts, T,
                       static_cast<const float*>(embed), static_cast<const float*>(gain), h,
                       static_cast<float*>(x), d, V, eps, err, kbM, pl, ctx, f, rope_cs);
  else
    hipLaunchKernelGGL(embed_norm_kernel<bf16_t>, grid, dim3(kNormThreads), 0, s, last, drafts, T,
                       static_cast<const bf16_t*>(embed), static_cast<const bf16_t*>(gain), h,
                       static_cast<bf16_t*>(x), d, V, eps, err, kbM, pl, ctx, f, rope_cs);
  return hipGetLastError();
}

hipError_t launch_embed_gather(const int32_t* last, const int32_t* drafts, int B, int T, const void* embed,
                               const void* gain, float* h, void* x, float* ssq, int d, int V, int* err,
                               const int32_t* ctx, float theta, float* rope_cs, hipStream_t s, const AttnPlan* plan) {
  RopeFreqHead f{};
  for (int j = 0; j < 64; ++j) f.inv_freq[j] = pow((double)theta, -2.0 * j / 128);
  const AttnPlan pl = plan ? *plan : AttnPlan{};
  hipLaunchKernelGGL(embed_gather_kernel, dim3(B * T + (pl.work ? 1 : 0)), dim3(kNormThreads), 0, s, last, drafts, T,
                     static_cast<const bf16_t*>(embed), static_cast<const bf16_t*>(gain), h, static_cast<bf16_t*>(x),
                     ssq, d, V, err, ctx, f, rope_cs, nullptr, pl);
  return hipGetLastError();
}

hipError_t launch_norm_inputs(const float* h, int B, int T, const void* gain, void* x, float* ssq, int d,
                              const int32_t* ctx, float theta, float* rope_cs, hipStream_t s) {
  RopeFreqHead f{};
  for (int j = 0; j < 64; ++j) f.inv_freq[j] = pow((double)theta, -2.0 * j / 128);
  hipLaunchKernelGGL(embed_gather_kernel, dim3(B * T), dim3(kNormThreads), 0, s, nullptr, nullptr, T, nullptr,
                     static_cast<const bf16_t*>(gain), nullptr, static_cast<bf16_t*>(x), ssq, d, 0, nullptr, ctx, f,
                     rope_cs, h, AttnPlan{});
  return hipGetLastError();
}

hipError_t launch_rmsnorm(int dtype, const float* h, const void* gain, void* x, int M, int d, float eps,
                          hipStream_t s, bool x_kblocked) {
  const int kbM = x_kblocked ? M : 0;
  if (dtype == kF32)
    hipLaunchKernelGGL(rmsnorm_kernel<float>, dim3(M), dim3(kNormThreads), 0, s, h,
                       static_cast<const float*>(gain), static_cast<float*>(x), d, eps, kbM);
  else
    hipLaunchKernelGGL(rmsnorm_kernel<bf16_t>, dim3(M), dim3(kNormThreads), 0, s, h,
                       static_cast<const bf16_t*>(gain), static_cast<bf16_t*>(x), d, eps, kbM);
  return hipGetLastError();
}

hipError_t launch_rope_window(int dtype, const float* qkv, const int32_t* ctx, int B, int T, int H, int Hkv, int D,
                              float theta, void* q_out, void* win_k, void* win_v, int32_t* ctx_snap, int* attn_counters,
                              hipStream_t s) {
  RopeFreq f{};
  const int half = D / 2;
  for (int j = 0; j < half && j < kMaxHalfDim; ++j) f.inv_freq[j] = pow((double)theta, -2.0 * j / D);
  if (dtype != kF32 && D == 128 && T <= kBlock) {
    hipLaunchKernelGGL(rope_window_d128_kernel, dim3(B, H + 2 * Hkv), dim3(256), 0, s, qkv, ctx, T, H, Hkv, f,
                       static_cast<bf16_t*>(q_out), static_cast<bf16_t*>(win_k), static_cast<bf16_t*>(win_v), ctx_snap,
                       attn_counters);
    return hipGetLastError();
  }
  const int hpb = half >= 256 ? 1 : 256 / half;
  dim3 grid(B * T, (H + 2 * Hkv + hpb - 1) / hpb), block(hpb * half);
  if (dtype == kF32)
    hipLaunchKernelGGL(rope_window_kernel<float>, grid, block, 0, s, qkv, ctx, T, H, Hkv, D, f,
                       static_cast<float*>(q_out), static_cast<float*>(win_k), static_cast<float*>(win_v), ctx_snap, attn_counters);
  else
    hipLaunchKernelGGL(rope_window_kernel<bf16_t>, grid, block, 0, s, qkv, ctx, T, H, Hkv, D, f,
                       static_cast<bf16_t*>(q_out), static_cast<bf16_t*>(win_k), static_cast<bf16_t*>(win_v), ctx_snap, attn_counters);
  return hipGetLastError();
}

hipError_t launch_kv_append(const KvAppendArgs& a, hipStream_t s) {
  const int ev = a.dtype == kF32 ? 4 : 8;
  const int pieces = (a.k + 1) * a.Hkv * (a.D / ev);
  for (int l0 = 0; l0 < a.L; l0 += kMaxAppendLayers) {
    const int nl = (a.L - l0 < kMaxAppendLayers) ? a.L - l0 : kMaxAppendLayers;
    const int last = l0 + nl == a.L;
    PagePtrs p{};
    for (int i = 0; i < nl; ++i) {
      p.k[i] = a.k_pages[l0 + i];
      p.v[i] = a.v_pages[l0 + i];
    }
    const dim3 grid((pieces + 255) / 256, a.B, nl);
    if (a.dtype == kF32)
      hipLaunchKernelGGL(kv_append_kernel<float>, grid, dim3(256), 0, s, p, l0, last,
                         static_cast<const float*>(a.win_k), static_cast<const float*>(a.win_v), a.block_table,
                         a.max_blocks, a.num_blocks, a.ctx_snap, a.ctx, a.accepted_len, a.B, a.k, a.Hkv, a.D, a.err);
    else
      hipLaunchKernelGGL(kv_append_kernel<bf16_t>, grid, dim3(256), 0, s, p, l0, last,
                         static_cast<const bf16_t*>(a.win_k), static_cast<const bf16_t*>(a.win_v), a.block_table,
                         a.max_blocks, a.num_blocks, a.ctx_snap, a.ctx, a.accepted_len, a.B, a.k, a.Hkv, a.D, a.err);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_copy_i32(int32_t* dst, const int32_t* src, int n, hipStream_t s) {
  hipLaunchKernelGGL(copy_i32_kernel, dim3((n + 255) / 256), dim3(256), 0, s, dst, src, n, 1);
  return hipGetLastError();
}

hipError_t launch_gather_u32(int32_t* dst, const int32_t* src, int n, int stride, hipStream_t s) {
  hipLaunchKernelGGL(copy_i32_kernel, dim3((n + 255) / 256), dim3(256), 0, s, dst, src, n, stride);
  return hipGetLastError();
}

hipError_t launch_fill_i32(int32_t* p, int32_t v, int n, hipStream_t s) {
  hipLaunchKernelGGL(fill_i32_kernel, dim3((n + 255) / 256), dim3(256), 0, s, p, v, n);
  return hipGetLastError();
}

}  // namespace nj
