// Small per-row kernels of the verify step: embedding gather fused with the
// first RMSNorm, RMSNorm, RoPE with the window K/V store, and the KV append
// of accepted rows.  All are HBM/latency bound and tiny next to the GEMMs.
#include "common.h"
#include "kernels.h"

namespace nj {
namespace {

constexpr int kNormThreads = 256;

// x = h / sqrt(mean(h^2) + eps) * gain, one row per workgroup.
template <typename T>
__device__ __forceinline__ void norm_row(const float* __restrict__ h, const T* __restrict__ gain,
                                         T* __restrict__ x, int d, float eps, float* sh) {
  float ss = 0.f;
  for (int i = threadIdx.x; i < d; i += kNormThreads) ss = fmaf(h[i], h[i], ss);
  ss = block_sum<kNormThreads>(ss, sh);
  const float r = 1.0f / sqrtf(ss / (float)d + eps);
  for (int i = threadIdx.x; i < d; i += kNormThreads) x[i] = from_f<T>(h[i] * r * to_f(gain[i]));
}

template <typename T>
__global__ __launch_bounds__(kNormThreads) void embed_norm_kernel(
    const int32_t* __restrict__ last, const int32_t* __restrict__ drafts, int T_, const T* __restrict__ embed,
    const T* __restrict__ gain, float* __restrict__ h, T* __restrict__ x, int d, int V, float eps,
    int* __restrict__ err) {
  __shared__ float sh[kNormThreads / kWave];
  const int row = blockIdx.x, b = row / T_, i = row % T_;
  int tok = (i == 0) ? last[b] : drafts[b * (T_ - 1) + i - 1];
  if (tok < 0 || tok >= V) {
    if (threadIdx.x == 0) flag_error(err, kErrToken);
    tok = 0;
  }
  const T* e = embed + (size_t)tok * d;
  float* hr = h + (size_t)row * d;
  for (int j = threadIdx.x; j < d; j += kNormThreads) hr[j] = to_f(e[j]);
  __syncthreads();
  norm_row<T>(hr, gain, x + (size_t)row * d, d, eps, sh);
}

template <typename T>
__global__ __launch_bounds__(kNormThreads) void rmsnorm_kernel(const float* __restrict__ h,
                                                               const T* __restrict__ gain, T* __restrict__ x,
                                                               int d, float eps) {
  __shared__ float sh[kNormThreads / kWave];
  norm_row<T>(h + (size_t)blockIdx.x * d, gain, x + (size_t)blockIdx.x * d, d, eps, sh);
}

// One workgroup per window row.  Pair (j, j + D/2) of every q and k head turns
// by pos * theta^(-2j/D), angle and sin/cos evaluated in fp64 (positions reach
// several thousand radians).  k goes to win_k[b][g][i][:], v to
// win_v[b][g][:][i]; the row i == 0 workgroup also zeroes the unused slots
// T..15 of the window block so that masked lanes never see stale data.
template <typename T>
__global__ __launch_bounds__(128) void rope_window_kernel(const float* __restrict__ qkv,
                                                          const int32_t* __restrict__ ctx, int T_, int H,
                                                          int Hkv, int D, float theta, T* __restrict__ q_out,
                                                          T* __restrict__ win_k, T* __restrict__ win_v) {
  const int row = blockIdx.x, b = row / T_, i = row % T_;
  const int half = D / 2;
  const double pos = (double)(max(ctx[b], 0) + i);
  const double ltheta = log((double)theta);
  const float* src = qkv + (size_t)row * (H + 2 * Hkv) * D;
  for (int idx = threadIdx.x; idx < (H + Hkv) * half; idx += blockDim.x) {
    const int hd = idx / half, j = idx % half;
    const double ang = pos * exp(-(2.0 * j / D) * ltheta);
    double sd, cd;
    sincos(ang, &sd, &cd);
    const float c = (float)cd, sn = (float)sd;
    const float a = src[hd * D + j], bb = src[hd * D + j + half];
    const float ra = a * c - bb * sn, rb = bb * c + a * sn;
    if (hd < H) {
      T* qo = q_out + ((size_t)row * H + hd) * D;
      qo[j] = from_f<T>(ra);
      qo[j + half] = from_f<T>(rb);
    } else {
      const int g = hd - H;
      T* ko = win_k + (((size_t)b * Hkv + g) * kBlock + i) * D;
      ko[j] = from_f<T>(ra);
      ko[j + half] = from_f<T>(rb);
    }
  }
  const float* vs = src + (H + Hkv) * D;
  for (int idx = threadIdx.x; idx < Hkv * D; idx += blockDim.x) {
    const int g = idx / D, dd = idx % D;
    win_v[(((size_t)b * Hkv + g) * D + dd) * kBlock + i] = from_f<T>(vs[idx]);
  }
  if (i == 0) {
    for (int idx = threadIdx.x; idx < Hkv * D * (kBlock - T_); idx += blockDim.x) {
      const int g = idx / (D * (kBlock - T_)), rem = idx % (D * (kBlock - T_));
      const int slot = T_ + rem / D, dd = rem % D;
      win_k[(((size_t)b * Hkv + g) * kBlock + slot) * D + dd] = from_f<T>(0.f);
      win_v[(((size_t)b * Hkv + g) * D + dd) * kBlock + slot] = from_f<T>(0.f);
    }
  }
}

constexpr int kMaxAppendLayers = 32;
struct PagePtrs {
  void* k[kMaxAppendLayers];
  void* v[kMaxAppendLayers];
};

// grid (B, layers of this chunk): copy window rows 0..n_b into their slots.
template <typename T>
__global__ __launch_bounds__(256) void kv_append_kernel(PagePtrs pages, int layer0, const T* __restrict__ win_k,
                                                        const T* __restrict__ win_v,
                                                        const int32_t* __restrict__ table, int max_blocks,
                                                        int num_blocks, const int32_t* __restrict__ ctx,
                                                        const int32_t* __restrict__ acc, int B, int k, int Hkv,
                                                        int D, int* __restrict__ err) {
  const int b = blockIdx.x, lc = blockIdx.y, l = layer0 + lc;
  const int n = acc[b], c = ctx[b];
  if (n < 0 || n > k) {
    if (threadIdx.x == 0) flag_error(err, kErrAccept);
    return;
  }
  if (c < 0 || c + k + 1 > max_blocks * kBlock) {
    if (threadIdx.x == 0) flag_error(err, kErrContext);
    return;
  }
  T* kp = static_cast<T*>(pages.k[lc]);
  T* vp = static_cast<T*>(pages.v[lc]);
  const size_t wbase = ((size_t)l * B + b) * Hkv;
  for (int j = 0; j <= n; ++j) {
    const int pos = c + j;
    const int phys = table[(size_t)b * max_blocks + pos / kBlock];
    if (phys < 0 || phys >= num_blocks) {
      if (threadIdx.x == 0) flag_error(err, kErrBlock);
      continue;
    }
    const int slot = pos % kBlock;
    for (int idx = threadIdx.x; idx < Hkv * D; idx += blockDim.x) {
      const int g = idx / D, dd = idx % D;
      kp[(((size_t)phys * Hkv + g) * kBlock + slot) * D + dd] = win_k[((wbase + g) * kBlock + j) * D + dd];
      vp[(((size_t)phys * Hkv + g) * D + dd) * kBlock + slot] = win_v[((wbase + g) * D + dd) * kBlock + j];
    }
  }
}

__global__ void ctx_update_kernel(int32_t* __restrict__ ctx, const int32_t* __restrict__ acc, int B, int k,
                                  int max_blocks) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  const int n = acc[b], c = ctx[b];
  if (n < 0 || n > k || c < 0 || c + k + 1 > max_blocks * kBlock) return;
  ctx[b] = c + n + 1;
}

__global__ void fill_i32_kernel(int32_t* p, int32_t v, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

}  // namespace

hipError_t launch_embed_norm(int dtype, const int32_t* last, const int32_t* drafts, int B, int T, const void* embed,
                             const void* gain, float* h, void* x, int d, int V, float eps, int* err,
                             hipStream_t s) {
  if (dtype == kF32)
    hipLaunchKernelGGL(embed_norm_kernel<float>, dim3(B * T), dim3(kNormThreads), 0, s, last, drafts, T,
                       static_cast<const float*>(embed), static_cast<const float*>(gain), h,
                       static_cast<float*>(x), d, V, eps, err);
  else
    hipLaunchKernelGGL(embed_norm_kernel<bf16_t>, dim3(B * T), dim3(kNormThreads), 0, s, last, drafts, T,
                       static_cast<const bf16_t*>(embed), static_cast<const bf16_t*>(gain), h,
                       static_cast<bf16_t*>(x), d, V, eps, err);
  return hipGetLastError();
}

hipError_t launch_rmsnorm(int dtype, const float* h, const void* gain, void* x, int M, int d, float eps,
                          hipStream_t s) {
  if (dtype == kF32)
    hipLaunchKernelGGL(rmsnorm_kernel<float>, dim3(M), dim3(kNormThreads), 0, s, h,
                       static_cast<const float*>(gain), static_cast<float*>(x), d, eps);
  else
    hipLaunchKernelGGL(rmsnorm_kernel<bf16_t>, dim3(M), dim3(kNormThreads), 0, s, h,
                       static_cast<const bf16_t*>(gain), static_cast<bf16_t*>(x), d, eps);
  return hipGetLastError();
}

hipError_t launch_rope_window(int dtype, const float* qkv, const int32_t* ctx, int B, int T, int H, int Hkv, int D,
                              float theta, void* q_out, void* win_k, void* win_v, hipStream_t s) {
  if (dtype == kF32)
    hipLaunchKernelGGL(rope_window_kernel<float>, dim3(B * T), dim3(128), 0, s, qkv, ctx, T, H, Hkv, D, theta,
                       static_cast<float*>(q_out), static_cast<float*>(win_k), static_cast<float*>(win_v));
  else
    hipLaunchKernelGGL(rope_window_kernel<bf16_t>, dim3(B * T), dim3(128), 0, s, qkv, ctx, T, H, Hkv, D, theta,
                       static_cast<bf16_t*>(q_out), static_cast<bf16_t*>(win_k), static_cast<bf16_t*>(win_v));
  return hipGetLastError();
}

hipError_t launch_kv_append(const KvAppendArgs& a, hipStream_t s) {
  for (int l0 = 0; l0 < a.L; l0 += kMaxAppendLayers) {
    const int nl = (a.L - l0 < kMaxAppendLayers) ? a.L - l0 : kMaxAppendLayers;
    PagePtrs p{};
    for (int i = 0; i < nl; ++i) {
      p.k[i] = a.k_pages[l0 + i];
      p.v[i] = a.v_pages[l0 + i];
    }
    if (a.dtype == kF32)
      hipLaunchKernelGGL(kv_append_kernel<float>, dim3(a.B, nl), dim3(256), 0, s, p, l0,
                         static_cast<const float*>(a.win_k), static_cast<const float*>(a.win_v), a.block_table,
                         a.max_blocks, a.num_blocks, a.ctx, a.accepted_len, a.B, a.k, a.Hkv, a.D, a.err);
    else
      hipLaunchKernelGGL(kv_append_kernel<bf16_t>, dim3(a.B, nl), dim3(256), 0, s, p, l0,
                         static_cast<const bf16_t*>(a.win_k), static_cast<const bf16_t*>(a.win_v),
                         a.block_table, a.max_blocks, a.num_blocks, a.ctx, a.accepted_len, a.B, a.k, a.Hkv, a.D,
                         a.err);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(ctx_update_kernel, dim3((a.B + 255) / 256), dim3(256), 0, s, a.ctx, a.accepted_len, a.B, a.k,
                     a.max_blocks);
  return hipGetLastError();
}

hipError_t launch_fill_i32(int32_t* p, int32_t v, int n, hipStream_t s) {
  hipLaunchKernelGGL(fill_i32_kernel, dim3((n + 255) / 256), dim3(256), 0, s, p, v, n);
  return hipGetLastError();
}

}  // namespace nj
