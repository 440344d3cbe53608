// Bandwidth-bound kernels of the decoder block, the embedding and the tied head.
// Storage type T is bf16 (bf16 workloads) or fp32; all arithmetic is fp32.
//
//  RMSNorm (App. E.2):   y = x r gamma, r = 1/sqrt(mean x^2 + eps)       one block per row
//  RMSNorm backward:     dx = resid + r (dn gamma - xhat mean(dn gamma xhat)),  dgamma partials
//  RoPE (rotate-half):   (a, b) <- (a cos - b sin, b cos + a sin), inverse with -sin
//  SwiGLU:               z = silu(a) b  (its backward runs in the down-projection GEMM epilogue)
//  Embedding:            x0[i] = E[tok[i]];  dE[v] = sum_{i: tok[i] = v} dx0[i] in position order
//  Cross-entropy:        dlogits = (softmax - onehot) * scale, row loss = lse - z[target]
#include "common.h"
#include "kernels.h"

namespace {

// ------------------------------------------------------------------ embedding gather
template <typename T>
__global__ void __launch_bounds__(256) embed_gather(const int32_t* __restrict__ tok,
                                                    const T* __restrict__ E, T* __restrict__ x0,
                                                    int d) {
  const int row = blockIdx.x;
  const int64_t src = (int64_t)tok[row] * d;
  const int64_t dst = (int64_t)row * d;
  for (int j = threadIdx.x; j < d; j += blockDim.x) x0[dst + j] = E[src + j];
}

// ------------------------------------------------------------------ RMSNorm
template <typename T>
__global__ void __launch_bounds__(256) rmsnorm_fwd(const T* __restrict__ x,
                                                   const T* __restrict__ gamma, T* __restrict__ y,
                                                   float* __restrict__ rstd, int d, float eps) {
  __shared__ float sm[16];
  const int64_t base = (int64_t)blockIdx.x * d;
  float ss = 0.f;
  for (int j = threadIdx.x; j < d; j += blockDim.x) {
    const float v = to_f32(x[base + j]);
    ss += v * v;
  }
  ss = block_sum<float>(ss, sm);
  const float r = 1.0f / sqrtf(ss / (float)d + eps);
  for (int j = threadIdx.x; j < d; j += blockDim.x)
    y[base + j] = from_f32<T>(to_f32(x[base + j]) * r * to_f32(gamma[j]));
  if (threadIdx.x == 0) rstd[blockIdx.x] = r;
}

// One block handles RMS_CHUNK consecutive rows; each thread owns columns j = tid + k*256 and
// keeps their dgamma partial sums in registers (d <= 256 * MAXC).
constexpr int MAXC = 16;
template <typename T>
__global__ void __launch_bounds__(256) rmsnorm_bwd(const T* __restrict__ dn, const T* __restrict__ x,
                                                   const float* __restrict__ rstd,
                                                   const T* __restrict__ gamma,
                                                   const T* __restrict__ resid, T* __restrict__ dx,
                                                   float* __restrict__ partial, int rows, int d) {
  __shared__ float sm[16];
  float dg[MAXC];
#pragma unroll
  for (int k = 0; k < MAXC; ++k) dg[k] = 0.f;
  const int r0 = blockIdx.x * RMS_CHUNK;
  const int r1 = min(rows, r0 + RMS_CHUNK);
  for (int r = r0; r < r1; ++r) {
    const int64_t base = (int64_t)r * d;
    const float rs = rstd[r];
    float dot = 0.f;
#pragma unroll
    for (int k = 0; k < MAXC; ++k) {
      const int j = threadIdx.x + k * 256;
      if (j < d) {
        const float xh = to_f32(x[base + j]) * rs;
        const float gv = to_f32(dn[base + j]);
        dot += gv * to_f32(gamma[j]) * xh;
        dg[k] += gv * xh;
      }
    }
    dot = block_sum<float>(dot, sm) / (float)d;
#pragma unroll
    for (int k = 0; k < MAXC; ++k) {
      const int j = threadIdx.x + k * 256;
      if (j < d) {
        const float xh = to_f32(x[base + j]) * rs;
        float v = rs * (to_f32(dn[base + j]) * to_f32(gamma[j]) - xh * dot);
        if (resid) v += to_f32(resid[base + j]);
        dx[base + j] = from_f32<T>(v);
      }
    }
  }
#pragma unroll
  for (int k = 0; k < MAXC; ++k) {
    const int j = threadIdx.x + k * 256;
    if (j < d) partial[(int64_t)blockIdx.x * d + j] = dg[k];
  }
}

// out[j] (+)= sum_c partial[c][j]: block of 1024 threads = 16 row groups x 64 columns; each thread
// sums rows g, g+16, ... of its column, then the 16 group sums are added in group order.
__global__ void __launch_bounds__(1024) colsum_partials(const float* __restrict__ partial,
                                                        int nchunks, int d, float* __restrict__ out,
                                                        int accumulate) {
  __shared__ float sm[16][64];
  const int c = threadIdx.x % 64, g = threadIdx.x / 64;
  const int j = blockIdx.x * 64 + c;
  float s = 0.f;
  if (j < d)
    for (int r = g; r < nchunks; r += 16) s += partial[(int64_t)r * d + j];
  sm[g][c] = s;
  __syncthreads();
  if (g == 0 && j < d) {
    float t = 0.f;
    for (int k = 0; k < 16; ++k) t += sm[k][c];
    out[j] = accumulate ? out[j] + t : t;
  }
}

// RMSNorm backward with one wave per row: lane l owns columns l + 64 k (k < CPL), gamma and the
// dgamma partial sums of those columns stay in registers, the row dot product is a wave reduction.
// Block = 4 waves over RMS_CHUNK consecutive rows; each wave writes its own dgamma partial row, so
// the partial array holds 4 rows per block.
template <typename T, int CPL>
__global__ void __launch_bounds__(256) rmsnorm_bwd_wave(const T* __restrict__ dn, const T* __restrict__ x,
                                                        const float* __restrict__ rstd,
                                                        const T* __restrict__ gamma,
                                                        const T* __restrict__ resid, T* __restrict__ dx,
                                                        float* __restrict__ partial, int rows) {
  constexpr int d = CPL * 64;
  const int wave = threadIdx.x / 64, lane = threadIdx.x % 64;
  float gm[CPL], dg[CPL];
#pragma unroll
  for (int k = 0; k < CPL; ++k) { gm[k] = to_f32(gamma[lane + 64 * k]); dg[k] = 0.f; }
  const int r0 = blockIdx.x * RMS_CHUNK;
  const int r1 = min(rows, r0 + RMS_CHUNK);
  for (int r = r0 + wave; r < r1; r += 4) {
    const int64_t base = (int64_t)r * d;
    const float rs = rstd[r];
    float xh[CPL], gv[CPL];
    float dot = 0.f;
#pragma unroll
    for (int k = 0; k < CPL; ++k) {
      xh[k] = to_f32(x[base + lane + 64 * k]) * rs;
      gv[k] = to_f32(dn[base + lane + 64 * k]);
      dot += gv[k] * gm[k] * xh[k];
      dg[k] += gv[k] * xh[k];
    }
    dot = wave_sum(dot) / (float)d;
#pragma unroll
    for (int k = 0; k < CPL; ++k) {
      float v = rs * (gv[k] * gm[k] - xh[k] * dot);
      if (resid) v += to_f32(resid[base + lane + 64 * k]);
      dx[base + lane + 64 * k] = from_f32<T>(v);
    }
  }
#pragma unroll
  for (int k = 0; k < CPL; ++k) partial[((int64_t)blockIdx.x * 4 + wave) * d + lane + 64 * k] = dg[k];
}

// ------------------------------------------------------------------ RoPE
template <typename T>
__global__ void __launch_bounds__(256) rope(T* __restrict__ qkv, int rows, int seq_len,
                                            int n_rot_heads, int hd, int ld,
                                            const float* __restrict__ ct,
                                            const float* __restrict__ st, float sgn) {
  const int half = hd / 2;
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t total = (int64_t)rows * n_rot_heads * half;
  if (idx >= total) return;
  const int i = idx % half;
  const int h = (idx / half) % n_rot_heads;
  const int row = idx / ((int64_t)half * n_rot_heads);
  const int p = row % seq_len;
  T* base = qkv + (int64_t)row * ld + h * hd;
  const float c = ct[p * half + i], s = sgn * st[p * half + i];
  const float a = to_f32(base[i]), b = to_f32(base[i + half]);
  base[i] = from_f32<T>(a * c - b * s);
  base[i + half] = from_f32<T>(b * c + a * s);
}

// ------------------------------------------------------------------ SwiGLU
__device__ __forceinline__ float sigm(float a) { return 1.0f / (1.0f + expf(-a)); }

template <typename T>
__global__ void __launch_bounds__(256) swiglu_fwd(const T* __restrict__ gu, T* __restrict__ z,
                                                  int rows, int f) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (int64_t)rows * f) return;
  const int64_t r = idx / f, j = idx % f;
  const float a = to_f32(gu[r * 2 * f + j]), b = to_f32(gu[r * 2 * f + f + j]);
  z[idx] = from_f32<T>(a * sigm(a) * b);
}

// ------------------------------------------------------------------ token sort (bitonic, LDS)
// keys (tok << 14) | pos are distinct, so the order is total; one block of 1024 threads.
constexpr int SORT_MAX = 16384;
__global__ void __launch_bounds__(1024) token_sort(const int32_t* __restrict__ tok, int n,
                                                   uint32_t* __restrict__ out) {
  __shared__ uint32_t k[SORT_MAX];
  int np = 1;
  while (np < n) np <<= 1;
  for (int i = threadIdx.x; i < np; i += blockDim.x)
    k[i] = i < n ? ((uint32_t)tok[i] << 14) | (uint32_t)i : 0xFFFFFFFFu;
  __syncthreads();
  for (int size = 2; size <= np; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int i = threadIdx.x; i < np; i += blockDim.x) {
        const int j = i ^ stride;
        if (j > i) {
          const bool up = (i & size) == 0;
          const uint32_t a = k[i], b = k[j];
          if ((a > b) == up) { k[i] = b; k[j] = a; }
        }
      }
      __syncthreads();
    }
  }
  for (int i = threadIdx.x; i < n; i += blockDim.x) out[i] = k[i];
}

// row_start[v] = first sorted index with token >= v (binary search), v in [0, vocab]
__global__ void __launch_bounds__(256) token_row_start(const uint32_t* __restrict__ sorted, int n,
                                                       int vocab, int32_t* __restrict__ row_start) {
  const int v = blockIdx.x * blockDim.x + threadIdx.x;
  if (v > vocab) return;
  int lo = 0, hi = n;
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if ((int)(sorted[mid] >> 14) < v) lo = mid + 1; else hi = mid;
  }
  row_start[v] = lo;
}

// ascending unique ids and counts from row_start; one block, each thread a contiguous id range
__global__ void __launch_bounds__(1024) token_compact(const int32_t* __restrict__ row_start,
                                                      int vocab, int32_t* __restrict__ ids,
                                                      int32_t* __restrict__ counts,
                                                      int32_t* __restrict__ n_unique) {
  __shared__ int32_t pre[1024];
  const int per = (vocab + blockDim.x - 1) / blockDim.x;
  const int lo = threadIdx.x * per, hi = min(vocab, lo + per);
  int c = 0;
  for (int v = lo; v < hi; ++v) c += row_start[v + 1] > row_start[v];
  pre[threadIdx.x] = c;
  __syncthreads();
  for (int off = 1; off < (int)blockDim.x; off <<= 1) {  // inclusive Hillis-Steele scan
    const int add = threadIdx.x >= off ? pre[threadIdx.x - off] : 0;
    __syncthreads();
    pre[threadIdx.x] += add;
    __syncthreads();
  }
  int o = pre[threadIdx.x] - c;
  for (int v = lo; v < hi; ++v) {
    const int cnt = row_start[v + 1] - row_start[v];
    if (cnt > 0) { ids[o] = v; counts[o] = cnt; ++o; }
  }
  if (threadIdx.x == blockDim.x - 1) n_unique[0] = pre[threadIdx.x];
}

// dE[v] (+)= sum over the run of v in position order; rows without tokens get 0 (overwrite)
template <typename T>
__global__ void __launch_bounds__(256) embed_scatter(const T* __restrict__ dx0,
                                                     const uint32_t* __restrict__ sorted,
                                                     const int32_t* __restrict__ row_start, int d,
                                                     float* __restrict__ de, int accumulate) {
  const int v = blockIdx.x;
  const int a = row_start[v], b = row_start[v + 1];
  if (accumulate && a == b) return;
  for (int j = threadIdx.x; j < d; j += blockDim.x) {
    float s = 0.f;
    for (int q = a; q < b; ++q) s += to_f32(dx0[(int64_t)(sorted[q] & 0x3FFFu) * d + j]);
    const int64_t o = (int64_t)v * d + j;
    de[o] = accumulate ? de[o] + s : s;
  }
}

// ------------------------------------------------------------------ cross-entropy rows
template <typename T>
__global__ void __launch_bounds__(256) ce_rows(const float* __restrict__ logits,
                                               const int32_t* __restrict__ tg, int V, float scale,
                                               T* __restrict__ dlog, float* __restrict__ row_loss) {
  __shared__ float sm[16];
  __shared__ float smx[16];
  const int64_t base = (int64_t)blockIdx.x * V;
  float mx = -INFINITY;
  for (int j = threadIdx.x; j < V; j += blockDim.x) mx = fmaxf(mx, logits[base + j]);
  mx = wave_max(mx);
  if (threadIdx.x % WAVE == 0) smx[threadIdx.x / WAVE] = mx;
  __syncthreads();
  mx = -INFINITY;
  for (int i = 0; i < (int)blockDim.x / WAVE; ++i) mx = fmaxf(mx, smx[i]);
  float se = 0.f;
  for (int j = threadIdx.x; j < V; j += blockDim.x) se += expf(logits[base + j] - mx);
  se = block_sum<float>(se, sm);
  const float lse = mx + logf(se);
  const int t = tg[blockIdx.x];
  for (int j = threadIdx.x; j < V; j += blockDim.x) {
    float p = expf(logits[base + j] - lse);
    if (j == t) p -= 1.0f;
    dlog[base + j] = from_f32<T>(p * scale);
  }
  if (threadIdx.x == 0) row_loss[blockIdx.x] = lse - logits[base + t];
}

__global__ void __launch_bounds__(1024) mean_kernel(const float* __restrict__ v, int n,
                                                    float* __restrict__ out) {
  __shared__ double sm[16];
  double s = 0.0;
  for (int i = threadIdx.x; i < n; i += blockDim.x) s += v[i];
  s = block_sum<double>(s, sm);
  if (threadIdx.x == 0) out[0] = (float)(s / n);
}

}  // namespace

#define DISPATCH(bf, KERNEL, ...) \
  do { if (bf) KERNEL<bf16>(__VA_ARGS__); else KERNEL<float>(__VA_ARGS__); } while (0)

template <typename T>
static void gather_t(const int32_t* tok, const void* E, void* x0, int rows, int d, hipStream_t st) {
  embed_gather<T><<<rows, 256, 0, st>>>(tok, (const T*)E, (T*)x0, d);
}
void launch_embed_gather(bool bf, const int32_t* tok, const void* table, void* x0, int rows, int d,
                         hipStream_t st) {
  DISPATCH(bf, gather_t, tok, table, x0, rows, d, st);
}

template <typename T>
static void rmsf_t(const void* x, const void* g, void* y, float* r, int rows, int d, float eps,
                   hipStream_t st) {
  rmsnorm_fwd<T><<<rows, 256, 0, st>>>((const T*)x, (const T*)g, (T*)y, r, d, eps);
}
void launch_rmsnorm_fwd(bool bf, const void* x, const void* gamma, void* y, float* rstd, int rows,
                        int d, float eps, hipStream_t st) {
  DISPATCH(bf, rmsf_t, x, gamma, y, rstd, rows, d, eps, st);
}

template <typename T>
static int rmsb_t(const void* dn, const void* x, const float* r, const void* g, const void* res,
                  void* dx, float* part, int rows, int d, hipStream_t st) {
  const unsigned nb = (unsigned)cdiv(rows, RMS_CHUNK);
#define RB(CPL) rmsnorm_bwd_wave<T, CPL><<<nb, 256, 0, st>>>((const T*)dn, (const T*)x, r, (const T*)g, \
                                                            (const T*)res, (T*)dx, part, rows)
  switch (d) {
    case 128: RB(2); return 4 * (int)nb;
    case 256: RB(4); return 4 * (int)nb;
    case 512: RB(8); return 4 * (int)nb;
    case 768: RB(12); return 4 * (int)nb;
    case 1024: RB(16); return 4 * (int)nb;
    case 2048: RB(32); return 4 * (int)nb;
    default: break;
  }
#undef RB
  rmsnorm_bwd<T><<<nb, 256, 0, st>>>((const T*)dn, (const T*)x, r, (const T*)g, (const T*)res, (T*)dx,
                                     part, rows, d);
  return (int)nb;
}
int launch_rmsnorm_bwd(bool bf, const void* dn, const void* x, const float* rstd,
                       const void* gamma, const void* resid, void* dx, float* partial, int rows,
                       int d, hipStream_t st) {
  return bf ? rmsb_t<bf16>(dn, x, rstd, gamma, resid, dx, partial, rows, d, st)
            : rmsb_t<float>(dn, x, rstd, gamma, resid, dx, partial, rows, d, st);
}

void launch_colsum_partials(const float* partial, int nchunks, int d, float* out, bool accumulate,
                            hipStream_t st) {
  colsum_partials<<<(unsigned)cdiv(d, 64), 1024, 0, st>>>(partial, nchunks, d, out,
                                                          accumulate ? 1 : 0);
}

template <typename T>
static void rope_t(void* qkv, int rows, int S, int nh, int hd, int ld, const float* c,
                   const float* s, bool inv, hipStream_t st) {
  const int64_t total = (int64_t)rows * nh * (hd / 2);
  rope<T><<<(unsigned)cdiv(total, 256), 256, 0, st>>>((T*)qkv, rows, S, nh, hd, ld, c, s,
                                                      inv ? -1.0f : 1.0f);
}
void launch_rope(bool bf, void* qkv, int rows, int seq_len, int n_rot_heads, int head_dim, int ld,
                 const float* cos_t, const float* sin_t, bool inverse, hipStream_t st) {
  DISPATCH(bf, rope_t, qkv, rows, seq_len, n_rot_heads, head_dim, ld, cos_t, sin_t, inverse, st);
}

template <typename T>
static void swf_t(const void* gu, void* z, int rows, int f, hipStream_t st) {
  swiglu_fwd<T><<<(unsigned)cdiv((int64_t)rows * f, 256), 256, 0, st>>>((const T*)gu, (T*)z, rows, f);
}
void launch_swiglu_fwd(bool bf, const void* gu, void* z, int rows, int f, hipStream_t st) {
  DISPATCH(bf, swf_t, gu, z, rows, f, st);
}
void launch_token_sort(const int32_t* tok, int n, uint32_t* sorted, hipStream_t st) {
  token_sort<<<1, 1024, 0, st>>>(tok, n, sorted);
}
void launch_token_runs(const uint32_t* sorted, int n, int vocab, int32_t* row_start, int32_t* ids,
                       int32_t* counts, int32_t* n_unique, hipStream_t st) {
  token_row_start<<<(unsigned)cdiv(vocab + 1, 256), 256, 0, st>>>(sorted, n, vocab, row_start);
  if (ids) token_compact<<<1, 1024, 0, st>>>(row_start, vocab, ids, counts, n_unique);
}
template <typename T>
static void scat_t(const void* dx0, const uint32_t* sorted, const int32_t* rs, int V, int d,
                   float* de, bool acc, hipStream_t st) {
  embed_scatter<T><<<V, 256, 0, st>>>((const T*)dx0, sorted, rs, d, de, acc ? 1 : 0);
}
void launch_embed_scatter(bool bf, const void* dx0, const uint32_t* sorted,
                          const int32_t* row_start, int vocab, int d, float* de, bool accumulate,
                          hipStream_t st) {
  DISPATCH(bf, scat_t, dx0, sorted, row_start, vocab, d, de, accumulate, st);
}

template <typename T>
static void ce_t(const float* logits, const int32_t* tg, int rows, int V, float scale, void* dl,
                 float* rl, hipStream_t st) {
  ce_rows<T><<<rows, 256, 0, st>>>(logits, tg, V, scale, (T*)dl, rl);
}
void launch_ce_rows(bool bf, const float* logits, const int32_t* targets, int rows, int vocab,
                    float scale, void* dlogits, float* row_loss, hipStream_t st) {
  DISPATCH(bf, ce_t, logits, targets, rows, vocab, scale, dlogits, row_loss, st);
}
void launch_mean(const float* v, int n, float* out, hipStream_t st) {
  mean_kernel<<<1, 1024, 0, st>>>(v, n, out);
}
