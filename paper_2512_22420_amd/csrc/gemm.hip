// GEMMs of the verify step: y = x . w^T over the B*(k+1) window rows.
//
// bf16 path: weight-streaming MFMA kernel.  At verify-step sizes M = B*(k+1)
// is 1..~768 while N*K reaches 5e8 (LM head), so below M ~ 300 the kernel is
// bound by reading each weight byte once from HBM.  Each wave owns 16 weight
// rows (the A operand of v_mfma_f32_16x16x32_bf16) and streams them along K
// with 16-byte loads, four 32-wide k-steps per pipeline stage, double
// buffered; the activation rows (B operand, M padded to 16) come from L2.
// Workgroups that would be too few to fill 256 CUs split K across their
// waves and reduce through LDS in a fixed order.  Epilogues: store fp32,
// residual add into the fp32 residual stream, SwiGLU into bf16 activations.
//
// Operand layout (16x16x32 bf16): lane l supplies row (l & 15) of A and
// column (l & 15) of B, eight consecutive k of k-group (l >> 4); the result
// lane l holds rows 4*(l >> 4) + i, column l & 15.  Any k permutation applied
// to both operands leaves the product unchanged.
#include "common.h"
#include "kernels.h"

namespace nj {
namespace {

constexpr int kU = 4;  // 32-wide k-steps per pipeline stage

__device__ __forceinline__ bf16x8 ld8(const bf16_t* p) {
  return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(p));
}

__device__ __forceinline__ float silu_mul(float gte, float up) { return gte / (1.0f + expf(-gte)) * up; }

// MT: 16-row tiles of x per workgroup; NG: weight row groups (2 for SwiGLU:
// gate rows n and up rows Nout + n); KSPLIT: waves sharing one 16-row weight
// tile along K; NW: waves per workgroup.
template <int MT, int NG, int KSPLIT, int NW, int EPI>
__global__ __launch_bounds__(NW * 64) void gemm_bf16_kernel(const bf16_t* __restrict__ X,
                                                            const bf16_t* __restrict__ W,
                                                            void* __restrict__ Y, int M, int Nout, int K) {
  constexpr int WN = NW / KSPLIT;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int ks = wave % KSPLIT, ns = wave / KSPLIT;
  const int r = lane & 15, g = lane >> 4;
  const int n0 = (blockIdx.x * WN + ns) * 16;
  const int m0 = blockIdx.y * (MT * 16);
  const bool active = n0 < Nout;

  const int nrow = min(n0 + r, Nout - 1);
  const bf16_t* wp[NG];
#pragma unroll
  for (int q = 0; q < NG; ++q) wp[q] = W + (size_t)(q * Nout + nrow) * K + g * 8;
  const bf16_t* xp[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) xp[mt] = X + (size_t)min(m0 + mt * 16 + r, M - 1) * K + g * 8;

  f32x4 acc[MT][NG];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int q = 0; q < NG; ++q) acc[mt][q] = f32x4{0.f, 0.f, 0.f, 0.f};

  if (active) {
    const int S = K / 32;
    const int s0 = (S * ks) / KSPLIT, s1 = (S * (ks + 1)) / KSPLIT;
    const int nfull = (s1 - s0) / kU;
    int s = s0;
    if (nfull > 0) {
      bf16x8 wa[NG][kU], xa[MT][kU];
#pragma unroll
      for (int u = 0; u < kU; ++u) {
#pragma unroll
        for (int q = 0; q < NG; ++q) wa[q][u] = ld8(wp[q] + (s + u) * 32);
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) xa[mt][u] = ld8(xp[mt] + (s + u) * 32);
      }
      for (int it = 0; it < nfull; ++it) {
        // prefetch the next stage (the last iteration re-reads its own stage)
        const int sn = (it + 1 < nfull) ? s + kU : s;
        bf16x8 wb[NG][kU], xb[MT][kU];
#pragma unroll
        for (int u = 0; u < kU; ++u) {
#pragma unroll
          for (int q = 0; q < NG; ++q) wb[q][u] = ld8(wp[q] + (sn + u) * 32);
#pragma unroll
          for (int mt = 0; mt < MT; ++mt) xb[mt][u] = ld8(xp[mt] + (sn + u) * 32);
        }
#pragma unroll
        for (int u = 0; u < kU; ++u)
#pragma unroll
          for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int q = 0; q < NG; ++q)
              acc[mt][q] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wa[q][u], xa[mt][u], acc[mt][q], 0, 0, 0);
#pragma unroll
        for (int u = 0; u < kU; ++u) {
#pragma unroll
          for (int q = 0; q < NG; ++q) wa[q][u] = wb[q][u];
#pragma unroll
          for (int mt = 0; mt < MT; ++mt) xa[mt][u] = xb[mt][u];
        }
        s += kU;
      }
    }
    for (; s < s1; ++s) {
      bf16x8 wv[NG], xv[MT];
#pragma unroll
      for (int q = 0; q < NG; ++q) wv[q] = ld8(wp[q] + s * 32);
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) xv[mt] = ld8(xp[mt] + s * 32);
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int q = 0; q < NG; ++q)
          acc[mt][q] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wv[q], xv[mt], acc[mt][q], 0, 0, 0);
    }
  }

  if constexpr (KSPLIT > 1) {
    __shared__ f32x4 red[NW][MT * NG][64];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int q = 0; q < NG; ++q) red[wave][mt * NG + q][lane] = acc[mt][q];
    __syncthreads();
    if (ks != 0) return;
    for (int k2 = 1; k2 < KSPLIT; ++k2)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int q = 0; q < NG; ++q) acc[mt][q] += red[wave + k2][mt * NG + q][lane];
  }
  if (!active) return;

  const int n = n0 + 4 * g;
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    const int m = m0 + mt * 16 + r;
    if (m >= M) continue;
    if constexpr (EPI == kEpiStore) {
      *reinterpret_cast<f32x4*>(static_cast<float*>(Y) + (size_t)m * Nout + n) = acc[mt][0];
    } else if constexpr (EPI == kEpiResidual) {
      f32x4* p = reinterpret_cast<f32x4*>(static_cast<float*>(Y) + (size_t)m * Nout + n);
      *p = *p + acc[mt][0];
    } else {
      const f32x4 a = acc[mt][0], b = acc[mt][1];
      u32x2 o;
      o[0] = pack_bf16x2(silu_mul(a[0], b[0]), silu_mul(a[1], b[1]));
      o[1] = pack_bf16x2(silu_mul(a[2], b[2]), silu_mul(a[3], b[3]));
      *reinterpret_cast<u32x2*>(static_cast<bf16_t*>(Y) + (size_t)m * Nout + n) = o;
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

template <int MT, int NG, int KSPLIT, int NW, int EPI>
hipError_t launch_bf16_cfg(const void* x, const void* w, void* y, int M, int Nout, int K, hipStream_t s) {
  constexpr int WN = NW / KSPLIT;
  const int ntiles = Nout / 16;
  dim3 grid((ntiles + WN - 1) / WN, (M + MT * 16 - 1) / (MT * 16));
  hipLaunchKernelGGL((gemm_bf16_kernel<MT, NG, KSPLIT, NW, EPI>), grid, dim3(NW * 64), 0, s,
                     static_cast<const bf16_t*>(x), static_cast<const bf16_t*>(w), y, M, Nout, K);
  return hipGetLastError();
}

template <int MT, int NG, int EPI>
hipError_t launch_bf16_mt(const void* x, const void* w, void* y, int M, int Nout, int K, int ksplit,
                          hipStream_t s) {
  switch (ksplit) {
    case 1: return launch_bf16_cfg<MT, NG, 1, 4, EPI>(x, w, y, M, Nout, K, s);
    case 2: return launch_bf16_cfg<MT, NG, 2, 4, EPI>(x, w, y, M, Nout, K, s);
    case 4: return launch_bf16_cfg<MT, NG, 4, 4, EPI>(x, w, y, M, Nout, K, s);
    default:
      if constexpr (NG == 1) return launch_bf16_cfg<MT, NG, 8, 8, EPI>(x, w, y, M, Nout, K, s);
      else return launch_bf16_cfg<MT, NG, 4, 4, EPI>(x, w, y, M, Nout, K, s);
  }
}

template <int NG, int EPI>
hipError_t launch_bf16_epi(const void* x, const void* w, void* y, int M, int Nout, int K, int mt, int ksplit,
                           hipStream_t s) {
  switch (mt) {
    case 1: return launch_bf16_mt<1, NG, EPI>(x, w, y, M, Nout, K, ksplit, s);
    case 2: return launch_bf16_mt<2, NG, EPI>(x, w, y, M, Nout, K, ksplit, s);
    case 3: return launch_bf16_mt<3, NG, EPI>(x, w, y, M, Nout, K, ksplit, s);
    default: return launch_bf16_mt<4, NG, EPI>(x, w, y, M, Nout, K, ksplit, s);
  }
}

}  // namespace

hipError_t launch_gemm(int dtype, const void* x, const void* w, void* y, int M, int N, int K, int epi,
                       hipStream_t s) {
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
  // bf16: 16-row x tiles per workgroup, then split K until ~2048 waves are in flight
  const int mt = M >= 64 ? 4 : (M + 15) / 16;
  const int mblocks = (M + mt * 16 - 1) / (mt * 16);
  const long tiles = (long)(Nout / 16) * mblocks;
  const int steps = K / 32;
  int ksplit = 1;
  while (ksplit < 8 && tiles * ksplit < 2048 && steps / (ksplit * 2) >= 8) ksplit *= 2;
  if (epi == kEpiSwiglu && ksplit > 4) ksplit = 4;
  if (epi == kEpiStore) return launch_bf16_epi<1, kEpiStore>(x, w, y, M, Nout, K, mt, ksplit, s);
  if (epi == kEpiResidual) return launch_bf16_epi<1, kEpiResidual>(x, w, y, M, Nout, K, mt, ksplit, s);
  return launch_bf16_epi<2, kEpiSwiglu>(x, w, y, M, Nout, K, mt, ksplit, s);
}

}  // namespace nj
