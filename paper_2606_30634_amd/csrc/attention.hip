// Causal grouped-query attention (App. E.2), reference tiling: one thread per query (forward,
// dQ) or key (dK, dV) row, K/V (or Q/dO) tiles of 64 rows staged through LDS, online softmax in
// fp32.  Used for fp32 workloads and shapes the MFMA kernels (attention_mfma.hip) do not take.
//
//   S = q k^T / sqrt(hd) on j <= i;  P = softmax(S);  o = P v;  lse_i = log sum_j exp(S_ij)
//   delta_i = sum_c dO_ic O_ic;  dP = dO v^T;  dS = P (dP - delta);  dq = dS k / sqrt(hd)
//   dk = dS^T q / sqrt(hd) and dv = P^T dO, summed over the query heads of a key/value head.
// Query head h reads key/value head h / (Hq / Hkv).
#include "common.h"
#include "kernels.h"

bool attention_mfma_fwd_try(const AttnArgs& a, hipStream_t st);  // attention_mfma.hip
bool attention_mfma_bwd_try(const AttnArgs& a, hipStream_t st);
bool attention_mfma_delta_try(const AttnArgs& a, hipStream_t st);

namespace {

constexpr int TR = 64;  // rows per block and per LDS tile

struct Geo {
  int ld, koff, voff, group;
  __device__ Geo(const AttnArgs& a) {
    ld = (a.Hq + 2 * a.Hkv) * a.hd;
    koff = a.Hq * a.hd;
    voff = (a.Hq + a.Hkv) * a.hd;
    group = a.Hq / a.Hkv;
  }
};

template <typename T, int HD>
__global__ void __launch_bounds__(TR) attn_fwd(AttnArgs a) {
  __shared__ float Ks[TR][HD];
  __shared__ float Vs[TR][HD];
  const Geo g(a);
  const int b = blockIdx.z, h = blockIdx.y, kvh = h / g.group;
  const int i = blockIdx.x * TR + threadIdx.x;
  const T* qkv = (const T*)a.qkv;
  const float scale = 1.0f / sqrtf((float)HD);
  float q[HD], o[HD];
  const int64_t rowq = (int64_t)(b * a.S + min(i, a.S - 1)) * g.ld;
#pragma unroll
  for (int c = 0; c < HD; ++c) { q[c] = to_f32(qkv[rowq + h * HD + c]) * scale; o[c] = 0.f; }
  float m = -INFINITY, l = 0.f;
  const int last = min(a.S - 1, blockIdx.x * TR + TR - 1);
  for (int j0 = 0; j0 <= last; j0 += TR) {
    __syncthreads();
    for (int e = threadIdx.x; e < TR * HD; e += TR) {
      const int r = e / HD, c = e % HD, j = j0 + r;
      const int64_t row = (int64_t)(b * a.S + min(j, a.S - 1)) * g.ld;
      Ks[r][c] = to_f32(qkv[row + g.koff + kvh * HD + c]);
      Vs[r][c] = to_f32(qkv[row + g.voff + kvh * HD + c]);
    }
    __syncthreads();
    const int jend = min(TR, i - j0 + 1);
    for (int r = 0; r < jend; ++r) {
      float s = 0.f;
#pragma unroll
      for (int c = 0; c < HD; ++c) s += q[c] * Ks[r][c];
      if (s > m) {
        const float corr = expf(m - s);
        l *= corr;
#pragma unroll
        for (int c = 0; c < HD; ++c) o[c] *= corr;
        m = s;
      }
      const float p = expf(s - m);
      l += p;
#pragma unroll
      for (int c = 0; c < HD; ++c) o[c] += p * Vs[r][c];
    }
  }
  if (i >= a.S) return;
  T* out = (T*)a.o;
  const int64_t rowo = (int64_t)(b * a.S + i) * a.Hq * HD + h * HD;
  const float inv = 1.0f / l;
#pragma unroll
  for (int c = 0; c < HD; ++c) out[rowo + c] = from_f32<T>(o[c] * inv);
  if (a.o32)
    for (int c = 0; c < HD; ++c) a.o32[rowo + c] = o[c] * inv;
  a.lse[((int64_t)b * a.Hq + h) * a.S + i] = m + logf(l);
}

// delta_i = sum_c dO_ic O_ic  (per query row and head)
template <typename T, int HD>
__global__ void __launch_bounds__(256) attn_delta(AttnArgs a) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;  // (b, h, i)
  if (idx >= (int64_t)a.B * a.Hq * a.S) return;
  const int i = idx % a.S, h = (idx / a.S) % a.Hq, b = idx / ((int64_t)a.S * a.Hq);
  const int64_t r = (int64_t)(b * a.S + i) * a.Hq * HD + h * HD;
  const T* dO = (const T*)a.dout;
  float s = 0.f;
  if (a.o32) {
    for (int c = 0; c < HD; ++c) s += a.o32[r + c] * to_f32(dO[r + c]);
  } else {
    const T* O = (const T*)a.o;
    for (int c = 0; c < HD; ++c) s += to_f32(O[r + c]) * to_f32(dO[r + c]);
  }
  a.delta[idx] = s;
}

// dq for query row i of head h
template <typename T, int HD>
__global__ void __launch_bounds__(TR) attn_bwd_dq(AttnArgs a) {
  __shared__ float Ks[TR][HD];
  __shared__ float Vs[TR][HD];
  const Geo g(a);
  const int b = blockIdx.z, h = blockIdx.y, kvh = h / g.group;
  const int i = blockIdx.x * TR + threadIdx.x;
  const int ic = min(i, a.S - 1);
  const T* qkv = (const T*)a.qkv;
  const T* dO = (const T*)a.dout;
  const float scale = 1.0f / sqrtf((float)HD);
  float q[HD], dq[HD], d_o[HD];
  const int64_t rowq = (int64_t)(b * a.S + ic) * g.ld;
  const int64_t rowo = (int64_t)(b * a.S + ic) * a.Hq * HD + h * HD;
#pragma unroll
  for (int c = 0; c < HD; ++c) {
    q[c] = to_f32(qkv[rowq + h * HD + c]) * scale;
    d_o[c] = to_f32(dO[rowo + c]);
    dq[c] = 0.f;
  }
  const int64_t sidx = ((int64_t)b * a.Hq + h) * a.S + ic;
  const float lse = a.lse[sidx], dl = a.delta[sidx];
  const int last = min(a.S - 1, blockIdx.x * TR + TR - 1);
  for (int j0 = 0; j0 <= last; j0 += TR) {
    __syncthreads();
    for (int e = threadIdx.x; e < TR * HD; e += TR) {
      const int r = e / HD, c = e % HD, j = j0 + r;
      const int64_t row = (int64_t)(b * a.S + min(j, a.S - 1)) * g.ld;
      Ks[r][c] = to_f32(qkv[row + g.koff + kvh * HD + c]);
      Vs[r][c] = to_f32(qkv[row + g.voff + kvh * HD + c]);
    }
    __syncthreads();
    const int jend = min(TR, i - j0 + 1);
    for (int r = 0; r < jend; ++r) {
      float s = 0.f, dp = 0.f;
#pragma unroll
      for (int c = 0; c < HD; ++c) { s += q[c] * Ks[r][c]; dp += d_o[c] * Vs[r][c]; }
      const float ds = expf(s - lse) * (dp - dl);
#pragma unroll
      for (int c = 0; c < HD; ++c) dq[c] += ds * Ks[r][c];
    }
  }
  if (i >= a.S) return;
  T* dqkv = (T*)a.dqkv;
#pragma unroll
  for (int c = 0; c < HD; ++c) dqkv[rowq + h * HD + c] = from_f32<T>(dq[c] * scale);
}

// dk (WANT_DK) or dv for key row j of key/value head kvh, summed over its query heads
template <typename T, int HD, bool WANT_DK>
__global__ void __launch_bounds__(TR) attn_bwd_dkv(AttnArgs a) {
  __shared__ float Qs[TR][HD];
  __shared__ float Ds[TR][HD];
  __shared__ float Ls[TR], Dl[TR];
  const Geo g(a);
  const int b = blockIdx.z, kvh = blockIdx.y;
  const int j = blockIdx.x * TR + threadIdx.x;
  const int jc = min(j, a.S - 1);
  const T* qkv = (const T*)a.qkv;
  const T* dO = (const T*)a.dout;
  const float scale = 1.0f / sqrtf((float)HD);
  float k[HD], v[HD], acc[HD];
  const int64_t rowk = (int64_t)(b * a.S + jc) * g.ld;
#pragma unroll
  for (int c = 0; c < HD; ++c) {
    k[c] = to_f32(qkv[rowk + g.koff + kvh * HD + c]);
    v[c] = WANT_DK ? to_f32(qkv[rowk + g.voff + kvh * HD + c]) : 0.f;
    acc[c] = 0.f;
  }
  const int first = blockIdx.x * TR;
  for (int hh = 0; hh < g.group; ++hh) {
    const int h = kvh * g.group + hh;
    for (int i0 = first; i0 < a.S; i0 += TR) {
      __syncthreads();
      for (int e = threadIdx.x; e < TR * HD; e += TR) {
        const int r = e / HD, c = e % HD, i = min(i0 + r, a.S - 1);
        Qs[r][c] = to_f32(qkv[(int64_t)(b * a.S + i) * g.ld + h * HD + c]) * scale;
        Ds[r][c] = to_f32(dO[(int64_t)(b * a.S + i) * a.Hq * HD + h * HD + c]);
      }
      {
        const int i = min(i0 + (int)threadIdx.x, a.S - 1);
        const int64_t sidx = ((int64_t)b * a.Hq + h) * a.S + i;
        Ls[threadIdx.x] = a.lse[sidx];
        Dl[threadIdx.x] = WANT_DK ? a.delta[sidx] : 0.f;
      }
      __syncthreads();
      const int rend = min(TR, a.S - i0);
      for (int r = 0; r < rend; ++r) {
        if (i0 + r < j) continue;  // causal: query i >= key j
        float s = 0.f;
#pragma unroll
        for (int c = 0; c < HD; ++c) s += Qs[r][c] * k[c];
        const float p = expf(s - Ls[r]);
        if (WANT_DK) {
          float dp = 0.f;
#pragma unroll
          for (int c = 0; c < HD; ++c) dp += Ds[r][c] * v[c];
          const float ds = p * (dp - Dl[r]);
#pragma unroll
          for (int c = 0; c < HD; ++c) acc[c] += ds * Qs[r][c];  // Qs already holds q * scale
        } else {
#pragma unroll
          for (int c = 0; c < HD; ++c) acc[c] += p * Ds[r][c];
        }
      }
    }
  }
  if (j >= a.S) return;
  T* dqkv = (T*)a.dqkv;
  const int off = WANT_DK ? g.koff : g.voff;
#pragma unroll
  for (int c = 0; c < HD; ++c) dqkv[rowk + off + kvh * HD + c] = from_f32<T>(acc[c]);
}

template <typename T, int HD>
void fwd_t(const AttnArgs& a, hipStream_t st) {
  attn_fwd<T, HD><<<dim3((unsigned)cdiv(a.S, TR), a.Hq, a.B), TR, 0, st>>>(a);
}
template <typename T, int HD>
void delta_t(const AttnArgs& a, hipStream_t st) {
  attn_delta<T, HD><<<(unsigned)cdiv((int64_t)a.B * a.Hq * a.S, 256), 256, 0, st>>>(a);
}
template <typename T, int HD>
void bwd_t(const AttnArgs& a, hipStream_t st) {
  if (!a.delta_ready) delta_t<T, HD>(a, st);
  attn_bwd_dq<T, HD><<<dim3((unsigned)cdiv(a.S, TR), a.Hq, a.B), TR, 0, st>>>(a);
  attn_bwd_dkv<T, HD, false><<<dim3((unsigned)cdiv(a.S, TR), a.Hkv, a.B), TR, 0, st>>>(a);
  attn_bwd_dkv<T, HD, true><<<dim3((unsigned)cdiv(a.S, TR), a.Hkv, a.B), TR, 0, st>>>(a);
}

template <typename T>
void fwd_hd(const AttnArgs& a, hipStream_t st) {
  if (a.hd == 32) fwd_t<T, 32>(a, st);
  else if (a.hd == 64) fwd_t<T, 64>(a, st);
  else fwd_t<T, 128>(a, st);
}
template <typename T>
void bwd_hd(const AttnArgs& a, hipStream_t st) {
  if (a.hd == 32) bwd_t<T, 32>(a, st);
  else if (a.hd == 64) bwd_t<T, 64>(a, st);
  else bwd_t<T, 128>(a, st);
}

}  // namespace

void launch_attention_fwd_ref(bool bf, const AttnArgs& a, hipStream_t st) {
  if (bf) fwd_hd<bf16>(a, st); else fwd_hd<float>(a, st);
}
void launch_attention_bwd_ref(bool bf, const AttnArgs& a, hipStream_t st) {
  if (bf) bwd_hd<bf16>(a, st); else bwd_hd<float>(a, st);
}

void launch_attention_fwd(bool bf, const AttnArgs& a, hipStream_t st) {
  if (bf && attention_mfma_fwd_try(a, st)) return;
  launch_attention_fwd_ref(bf, a, st);
}
void launch_attention_delta(bool bf, const AttnArgs& a, hipStream_t st) {
  if (bf && attention_mfma_delta_try(a, st)) return;
  auto run = [&](auto tag) {
    using T = decltype(tag);
    if (a.hd == 32) delta_t<T, 32>(a, st);
    else if (a.hd == 64) delta_t<T, 64>(a, st);
    else delta_t<T, 128>(a, st);
  };
  if (bf) run(bf16{}); else run(float{});
}

void launch_attention_bwd(bool bf, const AttnArgs& a, hipStream_t st) {
  if (bf && attention_mfma_bwd_try(a, st)) return;
  launch_attention_bwd_ref(bf, a, st);
  if (a.rope_cos)  // dq, dk back through the rotation (query heads and key heads are contiguous)
    launch_rope(bf, a.dqkv, a.B * a.S, a.S, a.Hq + a.Hkv, a.hd, (a.Hq + 2 * a.Hkv) * a.hd, a.rope_cos,
                a.rope_sin, true, st);
}
