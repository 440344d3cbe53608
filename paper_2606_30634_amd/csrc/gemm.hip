// GEMM entry: C[m, n] (+)= sum_k A(m, k) B(n, k) for the three products of a linear layer without
// bias (forward y = x W^T, input gradient dx = dy W, weight gradient dW = dy^T x).
//
// This file holds the reference tiling used for fp32 workloads and for shapes the MFMA kernel
// does not take: 64x64 output tile, 16-deep k slices staged through LDS, 4x4 outputs per
// thread, fp32 FMA.  bf16 workloads go to the MFMA kernel in gemm_mfma.hip.
#include "common.h"
#include "kernels.h"
#include <cstdio>
#include <cstdlib>

bool gemm_mfma_try(const GemmArgs& g, hipStream_t st);  // gemm_mfma.hip

namespace {

constexpr int TM = 64, TN = 64, TK = 16;

template <typename T, bool AK>
__device__ __forceinline__ float ldA(const T* A, int lda, int m, int k) {
  return to_f32(AK ? A[(int64_t)m * lda + k] : A[(int64_t)k * lda + m]);
}

template <typename T, typename OutT, bool AK, bool BK>
__global__ void __launch_bounds__(256) gemm_tiled(GemmArgs g) {
  __shared__ float As[TK][TM + 4];
  __shared__ float Bs[TK][TN + 4];
  const T* A = (const T*)g.A;
  const T* B = (const T*)g.B;
  const int m0 = blockIdx.y * TM, n0 = blockIdx.x * TN;
  const int tx = threadIdx.x % 16, ty = threadIdx.x / 16;
  float acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = 0.f;
  for (int k0 = 0; k0 < g.K; k0 += TK) {
    for (int e = threadIdx.x; e < TM * TK; e += 256) {
      int mm, kk;
      if (AK) { kk = e % TK; mm = e / TK; } else { mm = e % TM; kk = e / TM; }
      const int gm = m0 + mm, gk = k0 + kk;
      As[kk][mm] = (gm < g.M && gk < g.K) ? ldA<T, AK>(A, g.lda, gm, gk) : 0.f;
    }
    for (int e = threadIdx.x; e < TN * TK; e += 256) {
      int nn, kk;
      if (BK) { kk = e % TK; nn = e / TK; } else { nn = e % TN; kk = e / TN; }
      const int gn = n0 + nn, gk = k0 + kk;
      Bs[kk][nn] = (gn < g.N && gk < g.K) ? ldA<T, BK>(B, g.ldb, gn, gk) : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < TK; ++kk) {
      float a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = As[kk][ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = Bs[kk][tx * 4 + j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] += a[i] * b[j];
    }
    __syncthreads();
  }
  OutT* C = (OutT*)g.C;
  const T* R = (const T*)g.resid;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = m0 + ty * 4 + i;
    if (m >= g.M) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int n = n0 + tx * 4 + j;
      if (n >= g.N) continue;
      const int64_t o = (int64_t)m * g.ldc + n;
      float v = acc[i][j];
      if (g.epi == 1) {  // SwiGLU backward from dz = v
        const T* gu = (const T*)g.aux + (int64_t)m * g.ld_aux + n;
        const float a = to_f32(gu[0]), b = to_f32(gu[g.N]);
        const float sg = 1.0f / (1.0f + expf(-a));
        C[o] = from_f32<OutT>(v * b * sg * (1.0f + a * (1.0f - sg)));
        C[o + g.N] = from_f32<OutT>(v * a * sg);
        continue;
      }
      if (g.out_f32 && g.beta != 0.f) v += g.beta * to_f32(C[o]);
      if (R) v += to_f32(R[o]);
      C[o] = from_f32<OutT>(v);
    }
  }
}

template <typename T, typename OutT>
void launch_layout(const GemmArgs& g, hipStream_t st) {
  const dim3 grid((unsigned)cdiv(g.N, TN), (unsigned)cdiv(g.M, TM));
  if (g.a_kmajor && g.b_kmajor) gemm_tiled<T, OutT, true, true><<<grid, 256, 0, st>>>(g);
  else if (g.a_kmajor) gemm_tiled<T, OutT, true, false><<<grid, 256, 0, st>>>(g);
  else if (g.b_kmajor) gemm_tiled<T, OutT, false, true><<<grid, 256, 0, st>>>(g);
  else gemm_tiled<T, OutT, false, false><<<grid, 256, 0, st>>>(g);
}

}  // namespace

void launch_gemm_tiled(bool bf, const GemmArgs& g, hipStream_t st) {
  if (bf) {
    if (g.out_f32) launch_layout<bf16, float>(g, st);
    else launch_layout<bf16, bf16>(g, st);
  } else {
    launch_layout<float, float>(g, st);
  }
}

// y = alpha y + beta x, one thread per element of a rows x cols block of row stride ld
template <typename T>
__global__ void __launch_bounds__(256) axpby_kernel(T* __restrict__ y, const T* __restrict__ x, float alpha,
                                                    float beta, int rows, int cols, int ld) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (int64_t)rows * cols) return;
  const int64_t o = (i / cols) * ld + i % cols;
  y[o] = from_f32<T>(alpha * to_f32(y[o]) + beta * to_f32(x[o]));
}

void launch_axpby(bool bf, void* y, const void* x, float alpha, float beta, int rows, int cols, int ld,
                  hipStream_t st) {
  const unsigned nb = (unsigned)cdiv((int64_t)rows * cols, 256);
  if (bf) axpby_kernel<bf16><<<nb, 256, 0, st>>>((bf16*)y, (const bf16*)x, alpha, beta, rows, cols, ld);
  else axpby_kernel<float><<<nb, 256, 0, st>>>((float*)y, (const float*)x, alpha, beta, rows, cols, ld);
}

void launch_gemm(bool bf, const GemmArgs& g, hipStream_t st) {
  if (g.M == 0 || g.N == 0) return;
  if (bf && gemm_mfma_try(g, st)) return;
  if (g.epi == GEMM_EPI_AXPBY_DUP || g.epi == GEMM_EPI_NS_SPLIT) {
    // only the batched direct-to-LDS kernels implement these; callers check gemm_batched_tiles()
    fprintf(stderr, "launch_gemm: epilogue %d needs whole tiles and bf16 operands\n", g.epi);
    abort();
  }
  if (g.batch > 1 || g.epi == GEMM_EPI_AXPBY) {
    // one product at a time, then the AXPBY pass
    const size_t es = bf ? 2 : 4, cs = g.out_f32 ? 4 : es;
    for (int b = 0; b < g.batch; ++b) {
      GemmArgs p = g;
      p.batch = 1;
      p.A = (const char*)g.A + b * g.sA * es;
      p.B = (const char*)g.B + b * g.sB * es;
      p.C = (char*)g.C + b * g.sC * cs;
      p.D = g.D ? (const char*)g.D + b * g.sD * cs : nullptr;
      if (g.epi == GEMM_EPI_AXPBY) {
        p.epi = 0;
        launch_gemm(bf, p, st);
        launch_axpby(bf && !g.out_f32, p.C, p.D, g.alpha, g.beta_d, g.M, g.N, g.ldc, st);
      } else {
        launch_gemm(bf, p, st);
      }
    }
    return;
  }
  if (g.epi == 4) {  // the product, then delta = rowsum(dO O) by the attention's own kernel
    GemmArgs p = g;
    p.epi = 0;
    launch_gemm(bf, p, st);
    AttnArgs a{};
    a.B = g.M / g.delta_S; a.S = g.delta_S; a.Hq = g.N / g.delta_hd; a.Hkv = a.Hq; a.hd = g.delta_hd;
    a.o = const_cast<void*>(g.aux); a.o32 = (float*)const_cast<void*>(g.aux);  // O in fp32
    a.dout = g.C; a.delta = g.delta;
    launch_attention_delta(bf, a, st);
    return;
  }
  if (g.epi == 3) {  // the reference tiling writes gate|up, then the SwiGLU kernel makes z
    GemmArgs p = g;
    p.epi = 0;
    p.glu = 0;
    launch_gemm_tiled(bf, p, st);
    launch_swiglu_fwd(bf, g.C, g.out2, g.M, g.glu, st);
    return;
  }
  if (g.epi == 2) {  // the reference tiling writes the products, then the rotation runs
    GemmArgs p = g;
    p.epi = 0;
    launch_gemm_tiled(bf, p, st);
    launch_rope(bf, g.C, g.M, g.rope_S, g.rope_cols / g.rope_hd, g.rope_hd, g.ldc, g.rope_cos, g.rope_sin,
                false, st);
    return;
  }
  launch_gemm_tiled(bf, g, st);
}
