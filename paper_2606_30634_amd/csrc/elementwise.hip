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
// A token outside [0, vocab) embeds as a zero row.
template <typename T>
__global__ void __launch_bounds__(256) embed_gather(const int32_t* __restrict__ tok,
                                                    const T* __restrict__ E, T* __restrict__ x0,
                                                    int d, int vocab) {
  const int row = blockIdx.x;
  const int t = tok[row];
  const bool ok = t >= 0 && t < vocab;
  const int64_t src = (int64_t)(ok ? t : 0) * d;
  const int64_t dst = (int64_t)row * d;
  for (int j = threadIdx.x; j < d; j += blockDim.x) x0[dst + j] = ok ? E[src + j] : from_f32<T>(0.f);
}

// The same in 16-byte chunks, one wave per row and four rows per block (d a multiple of the
// chunk, table and output 16-byte aligned).
template <typename T>
__global__ void __launch_bounds__(256) embed_gather_vec(const int32_t* __restrict__ tok,
                                                        const T* __restrict__ E, T* __restrict__ x0,
                                                        int rows, int d, int vocab) {
  constexpr int V = 16 / (int)sizeof(T);
  const int row = blockIdx.x * 4 + threadIdx.x / 64, lane = threadIdx.x % 64;
  if (row >= rows) return;
  const int t = tok[row];
  const bool ok = t >= 0 && t < vocab;
  const uint4* src = reinterpret_cast<const uint4*>(E + (int64_t)(ok ? t : 0) * d);
  uint4* dst = reinterpret_cast<uint4*>(x0 + (int64_t)row * d);
  const int nc = d / V;
  for (int c = lane; c < nc; c += 64) dst[c] = ok ? src[c] : make_uint4(0u, 0u, 0u, 0u);
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

// Fixed-order column sums of a [nrows][d] fp32 array, one level of a two-level tree: thread j of
// group g sums rows [g G, min(g G + G, nrows)) of column j in row order and writes dst[g][j]
// (dst (+)= when accumulate, used for the last level whose single group covers every row).
__global__ void __launch_bounds__(256) colsum_rows(const float* __restrict__ src, int nrows, int d, int G,
                                                   float* __restrict__ dst, int accumulate) {
  const int j = blockIdx.x * 256 + threadIdx.x;
  if (j >= d) return;
  const int r0 = blockIdx.y * G, r1 = min(nrows, r0 + G);
  float s = 0.f;
#pragma unroll 8
  for (int r = r0; r < r1; ++r) s += src[(int64_t)r * d + j];
  float* o = dst + (int64_t)blockIdx.y * d + j;
  *o = accumulate ? *o + s : s;
}

template <typename T, int V>
struct Vec {
  typedef T type __attribute__((ext_vector_type(V)));
};

// RMSNorm backward, one wave per row and U rows in flight per wave: lane l owns the V-element
// vectors at columns (l + 64 k) V, k < NI, so every load and store is V elements wide; gamma and
// the dgamma partial sums of those columns stay in registers and the row dot product is a wave
// reduction.  A block covers RMS_ROWS_VEC consecutive rows (4 per wave) and writes one dgamma
// partial row, the sum of its waves' rows in wave order.
constexpr int RMS_ROWS_VEC = 16;
// RMSNorm forward, one wave per row and two rows in flight per wave: lane l owns the V-element
// vectors at columns (l + 64 k) V, k < NI, keeps gamma of those columns in registers for all its
// rows, and the row's sum of squares is a wave reduction.  A block covers RMS_ROWS_VEC
// consecutive rows (rows wave, wave + 4, ... of the block).
template <typename T, int V, int NI>
__global__ void __launch_bounds__(256) rmsnorm_fwd_vec(const T* __restrict__ x, const T* __restrict__ gamma,
                                                       T* __restrict__ y, float* __restrict__ rstd,
                                                       int rows, float eps) {
  constexpr int d = 64 * V * NI;
  using VT = typename Vec<T, V>::type;
  const int wave = threadIdx.x / 64, lane = threadIdx.x % 64;
  float gm[NI][V];
#pragma unroll
  for (int k = 0; k < NI; ++k) {
    const VT gv = *reinterpret_cast<const VT*>(gamma + (lane + 64 * k) * V);
#pragma unroll
    for (int q = 0; q < V; ++q) gm[k][q] = to_f32(gv[q]);
  }
  const int r0 = blockIdx.x * RMS_ROWS_VEC + wave;
#pragma unroll 1
  for (int it = 0; it < RMS_ROWS_VEC / 8; ++it) {
    int r[2];
    VT xv[2][NI];
    float ss[2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      r[u] = r0 + 4 * (2 * it + u);
      const int64_t base = (int64_t)(r[u] < rows ? r[u] : 0) * d;
#pragma unroll
      for (int k = 0; k < NI; ++k) xv[u][k] = *reinterpret_cast<const VT*>(x + base + (lane + 64 * k) * V);
    }
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      ss[u] = 0.f;
#pragma unroll
      for (int k = 0; k < NI; ++k)
#pragma unroll
        for (int q = 0; q < V; ++q) {
          const float v = to_f32(xv[u][k][q]);
          ss[u] += v * v;
        }
    }
#pragma unroll
    for (int u = 0; u < 2; ++u) ss[u] = wave_sum(ss[u]);
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      if (r[u] >= rows) continue;
      const float rs = 1.0f / sqrtf(ss[u] / (float)d + eps);
      const int64_t base = (int64_t)r[u] * d;
#pragma unroll
      for (int k = 0; k < NI; ++k) {
        VT ov;
#pragma unroll
        for (int q = 0; q < V; ++q) ov[q] = from_f32<T>(to_f32(xv[u][k][q]) * rs * gm[k][q]);
        *reinterpret_cast<VT*>(y + base + (lane + 64 * k) * V) = ov;
      }
      if (lane == 0) rstd[r[u]] = rs;
    }
  }
}

template <typename T, int V, int NI>
__global__ void __launch_bounds__(256) rmsnorm_bwd_vec(const T* __restrict__ dn, const T* __restrict__ x,
                                                       const float* __restrict__ rstd,
                                                       const T* __restrict__ gamma,
                                                       const T* __restrict__ resid, T* __restrict__ dx,
                                                       float* __restrict__ partial, int rows) {
  constexpr int d = 64 * V * NI;
  constexpr int U = V * NI <= 12 ? 2 : 1;  // two rows in flight while registers allow
  using VT = typename Vec<T, V>::type;
  __shared__ float red[d];
  const int wave = threadIdx.x / 64, lane = threadIdx.x % 64;
  float gm[NI][V], dg[NI][V];
#pragma unroll
  for (int k = 0; k < NI; ++k) {
    const VT gv = *reinterpret_cast<const VT*>(gamma + (lane + 64 * k) * V);
#pragma unroll
    for (int q = 0; q < V; ++q) { gm[k][q] = to_f32(gv[q]); dg[k][q] = 0.f; }
  }
  const int r0 = blockIdx.x * RMS_ROWS_VEC + wave;
#pragma unroll 1
  for (int it = 0; it < RMS_ROWS_VEC / (4 * U); ++it) {
    int r[U];
    bool ok[U];
    VT xv[U][NI], gv[U][NI], rv[U][NI];
    float rs[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      r[u] = r0 + 4 * (U * it + u);
      ok[u] = r[u] < rows;
      const int64_t base = (int64_t)(ok[u] ? r[u] : 0) * d;
      rs[u] = ok[u] ? rstd[r[u]] : 0.f;
#pragma unroll
      for (int k = 0; k < NI; ++k) {
        const int64_t o = base + (lane + 64 * k) * V;
        xv[u][k] = *reinterpret_cast<const VT*>(x + o);
        gv[u][k] = *reinterpret_cast<const VT*>(dn + o);
        if (resid) rv[u][k] = *reinterpret_cast<const VT*>(resid + o);
      }
    }
    float dot[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      dot[u] = 0.f;
#pragma unroll
      for (int k = 0; k < NI; ++k)
#pragma unroll
        for (int q = 0; q < V; ++q) {
          const float xh = to_f32(xv[u][k][q]) * rs[u], g = to_f32(gv[u][k][q]);
          dot[u] += g * gm[k][q] * xh;
          dg[k][q] += g * xh;  // rs = 0 on a row past the end adds nothing
        }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) dot[u] = wave_sum(dot[u]) / (float)d;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (!ok[u]) continue;
      const int64_t base = (int64_t)r[u] * d;
#pragma unroll
      for (int k = 0; k < NI; ++k) {
        VT ov;
#pragma unroll
        for (int q = 0; q < V; ++q) {
          const float xh = to_f32(xv[u][k][q]) * rs[u];
          float v = rs[u] * (to_f32(gv[u][k][q]) * gm[k][q] - xh * dot[u]);
          if (resid) v += to_f32(rv[u][k][q]);
          ov[q] = from_f32<T>(v);
        }
        *reinterpret_cast<VT*>(dx + base + (lane + 64 * k) * V) = ov;
      }
    }
  }
  // dgamma partial of the block: wave 0's sums, then waves 1, 2, 3 added in that order
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    if (wave == w)
#pragma unroll
      for (int k = 0; k < NI; ++k)
#pragma unroll
        for (int q = 0; q < V; ++q) {
          float& e = red[(lane + 64 * k) * V + q];
          e = (w == 0 ? 0.f : e) + dg[k][q];
        }
    __syncthreads();
  }
  for (int c = threadIdx.x; c < d; c += 256) partial[(int64_t)blockIdx.x * d + c] = red[c];
}

// RMSNorm backward for wide rows (d = 4 * 64 * V * NI >= 2048): the block's four waves split
// every row's columns, so a lane holds V * NI gains and dgamma sums instead of the whole row's
// share; the row's dot product is the four wave sums added in wave order through LDS (two rows
// in flight, a double-buffered exchange, one barrier per pair).  Each wave's dgamma columns are
// its own: the block's partial row is written without a cross-wave reduction.
template <typename T, int V, int NI>
__global__ void __launch_bounds__(256) rmsnorm_bwd_slice(const T* __restrict__ dn, const T* __restrict__ x,
                                                         const float* __restrict__ rstd,
                                                         const T* __restrict__ gamma,
                                                         const T* __restrict__ resid, T* __restrict__ dx,
                                                         float* __restrict__ partial, int rows) {
  constexpr int W = 64 * V * NI, d = 4 * W, U = 2;
  static_assert(RMS_ROWS_VEC % U == 0, "row pairs");
  using VT = typename Vec<T, V>::type;
  __shared__ float sdot[2][U][4];
  const int wave = threadIdx.x / 64, lane = threadIdx.x % 64;
  const int c0 = wave * W;
  float gm[NI][V], dg[NI][V];
#pragma unroll
  for (int k = 0; k < NI; ++k) {
    const VT gv = *reinterpret_cast<const VT*>(gamma + c0 + (lane + 64 * k) * V);
#pragma unroll
    for (int q = 0; q < V; ++q) { gm[k][q] = to_f32(gv[q]); dg[k][q] = 0.f; }
  }
#pragma unroll 1
  for (int it = 0; it < RMS_ROWS_VEC / U; ++it) {
    int r[U];
    bool ok[U];
    VT xv[U][NI], gv[U][NI], rv[U][NI];
    float rs[U], dot[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      r[u] = blockIdx.x * RMS_ROWS_VEC + U * it + u;
      ok[u] = r[u] < rows;
      const int64_t base = (int64_t)(ok[u] ? r[u] : 0) * d + c0;
      rs[u] = ok[u] ? rstd[r[u]] : 0.f;
#pragma unroll
      for (int k = 0; k < NI; ++k) {
        const int64_t o = base + (lane + 64 * k) * V;
        xv[u][k] = *reinterpret_cast<const VT*>(x + o);
        gv[u][k] = *reinterpret_cast<const VT*>(dn + o);
        if (resid) rv[u][k] = *reinterpret_cast<const VT*>(resid + o);
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      dot[u] = 0.f;
#pragma unroll
      for (int k = 0; k < NI; ++k)
#pragma unroll
        for (int q = 0; q < V; ++q) {
          const float xh = to_f32(xv[u][k][q]) * rs[u], g = to_f32(gv[u][k][q]);
          dot[u] += g * gm[k][q] * xh;
          dg[k][q] += g * xh;  // rs = 0 on a row past the end adds nothing
        }
      dot[u] = wave_sum(dot[u]);
    }
    const int buf = it & 1;
    if (lane == 0) {
#pragma unroll
      for (int u = 0; u < U; ++u) sdot[buf][u][wave] = dot[u];
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < U; ++u)
      dot[u] = (((sdot[buf][u][0] + sdot[buf][u][1]) + sdot[buf][u][2]) + sdot[buf][u][3]) / (float)d;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (!ok[u]) continue;
      const int64_t base = (int64_t)r[u] * d + c0;
#pragma unroll
      for (int k = 0; k < NI; ++k) {
        VT ov;
#pragma unroll
        for (int q = 0; q < V; ++q) {
          const float xh = to_f32(xv[u][k][q]) * rs[u];
          float v = rs[u] * (to_f32(gv[u][k][q]) * gm[k][q] - xh * dot[u]);
          if (resid) v += to_f32(rv[u][k][q]);
          ov[q] = from_f32<T>(v);
        }
        *reinterpret_cast<VT*>(dx + base + (lane + 64 * k) * V) = ov;
      }
    }
  }
#pragma unroll
  for (int k = 0; k < NI; ++k)
#pragma unroll
    for (int q = 0; q < V; ++q) partial[(int64_t)blockIdx.x * d + c0 + (lane + 64 * k) * V + q] = dg[k][q];
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

// ------------------------------------------------------------------ token sort (radix sort)
// Positions sorted by token, stably (equal tokens keep ascending positions): an LSD radix sort of the
// keys key_i = token_i (tokens outside [0, vocab) keyed as vocab, so that they sort after every valid
// one and belong to no embedding row; vocab < 2^17) carrying the positions, in three passes of 6-bit
// digits.  A pass: per chunk of RADIX_CHUNK consecutive keys the digit counts (one wave walks the
// chunk in rounds of 64 keys); one exclusive scan over (digit, chunk) in digit-major order; then the
// stable scatter, where a key's place is its (digit, chunk) offset plus the number of keys with the
// same digit before it in the chunk.  Within a round, the lanes holding a digit find each other from
// six ballots of the digit's bits; the lowest of them advances the digit's running offset.  Integer
// counts in a fixed order: the result is the same on every run.
constexpr int RADIX_CHUNK = 1024, RADIX_BITS = 6, RADIX_DIG = 1 << RADIX_BITS, RADIX_PASSES = 3;
__device__ __forceinline__ uint32_t token_key(const int32_t* tok, int i, int vocab) {
  const int t = tok[i];
  return (uint32_t)(t >= 0 && t < vocab ? t : vocab);
}
// lanes of the wave whose digit equals this lane's (among the active ones)
__device__ __forceinline__ uint64_t digit_match(uint32_t dig, uint64_t active) {
  uint64_t m = active;
#pragma unroll
  for (int b = 0; b < RADIX_BITS; ++b) {
    const uint64_t bal = __ballot((dig >> b) & 1u);
    m &= ((dig >> b) & 1u) ? bal : ~bal;
  }
  return m;
}
// keys of pass 0 from the tokens (vals = positions), later passes from the previous pass's output
__device__ __forceinline__ uint32_t radix_in(const int32_t* tok, const uint32_t* keys, int i, int vocab) {
  return tok ? token_key(tok, i, vocab) : keys[i];
}
__global__ void __launch_bounds__(64) radix_count(const int32_t* __restrict__ tok, const uint32_t* __restrict__ keys,
                                                  int n, int vocab, int shift, int nchunk, int32_t* __restrict__ hist) {
  __shared__ int cnt[RADIX_DIG];
  const int lane = threadIdx.x;
  cnt[lane] = 0;  // RADIX_DIG == the wave's 64 lanes
  __syncthreads();
  const int c0 = blockIdx.x * RADIX_CHUNK, c1 = min(n, c0 + RADIX_CHUNK);
  for (int r = c0; r < c1; r += 64) {
    const int i = r + lane;
    const bool on = i < c1;
    const uint32_t dig = on ? (radix_in(tok, keys, i, vocab) >> shift) & (RADIX_DIG - 1) : 0u;
    const uint64_t m = digit_match(dig, __ballot(on));
    if (on && (m & ((1ull << lane) - 1)) == 0) cnt[dig] += __popcll(m);  // the digit's lowest lane
    __syncthreads();
  }
  hist[(int64_t)lane * nchunk + blockIdx.x] = cnt[lane];
}
// exclusive scan of hist [RADIX_DIG][nchunk] in place, one block
__global__ void __launch_bounds__(1024) radix_scan(int32_t* __restrict__ hist, int total) {
  __shared__ int32_t part[1024];
  const int per = (total + blockDim.x - 1) / blockDim.x;
  const int lo = threadIdx.x * per, hi = min(total, lo + per);
  int c = 0;
  for (int q = lo; q < hi; ++q) c += hist[q];
  part[threadIdx.x] = c;
  __syncthreads();
  for (int off = 1; off < (int)blockDim.x; off <<= 1) {  // inclusive Hillis-Steele scan
    const int add = threadIdx.x >= off ? part[threadIdx.x - off] : 0;
    __syncthreads();
    part[threadIdx.x] += add;
    __syncthreads();
  }
  int o = part[threadIdx.x] - c;
  for (int q = lo; q < hi; ++q) {
    const int v = hist[q];
    hist[q] = o;
    o += v;
  }
}
__global__ void __launch_bounds__(64) radix_scatter(const int32_t* __restrict__ tok, const uint32_t* __restrict__ keys,
                                                    const uint32_t* __restrict__ vals, int n, int vocab, int shift,
                                                    int nchunk, const int32_t* __restrict__ offs,
                                                    uint32_t* __restrict__ keys_out, uint32_t* __restrict__ vals_out) {
  __shared__ int base[RADIX_DIG];
  const int lane = threadIdx.x;
  base[lane] = offs[(int64_t)lane * nchunk + blockIdx.x];
  __syncthreads();
  const int c0 = blockIdx.x * RADIX_CHUNK, c1 = min(n, c0 + RADIX_CHUNK);
  for (int r = c0; r < c1; r += 64) {
    const int i = r + lane;
    const bool on = i < c1;
    const uint32_t key = on ? radix_in(tok, keys, i, vocab) : 0u;
    const uint32_t dig = (key >> shift) & (RADIX_DIG - 1);
    const uint64_t m = digit_match(dig, __ballot(on));
    const int rank = __popcll(m & ((1ull << lane) - 1));
    const int dst = on ? base[dig] + rank : 0;
    __syncthreads();  // every lane has read its digit's offset before the offsets move on
    if (on) {
      keys_out[dst] = key;
      vals_out[dst] = tok ? (uint32_t)i : vals[i];
      if (rank == 0) base[dig] += __popcll(m);
    }
    __syncthreads();
  }
}

// row_start[v] = first sorted index with token >= v (binary search over the sorted tokens), v in [0, vocab]
__global__ void __launch_bounds__(256) token_row_start(const uint32_t* __restrict__ sorted_tok, int n,
                                                       int vocab, int32_t* __restrict__ row_start) {
  const int v = blockIdx.x * blockDim.x + threadIdx.x;
  if (v > vocab) return;
  int lo = 0, hi = n;
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if ((int)sorted_tok[mid] < v) lo = mid + 1; else hi = mid;
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
                                                     const uint32_t* __restrict__ sorted_pos,
                                                     const int32_t* __restrict__ row_start, int d,
                                                     float* __restrict__ de, int accumulate) {
  const int v = blockIdx.x;
  const int a = row_start[v], b = row_start[v + 1];
  if (accumulate && a == b) return;
  for (int j = threadIdx.x; j < d; j += blockDim.x) {
    float s = 0.f;
    for (int q = a; q < b; ++q) s += to_f32(dx0[(int64_t)sorted_pos[q] * d + j]);
    const int64_t o = (int64_t)v * d + j;
    de[o] = accumulate ? de[o] + s : s;
  }
}

// ------------------------------------------------------------------ cross-entropy rows
// Cross-entropy of one row of logits z [V] (one block per row), in two passes over the fp32
// logits: the forward keeps a running (max m, sum s of exp(z - m)) per thread over 16-byte
// chunks, merges the pairs across the block in a fixed order and writes lse = m + log s and the
// row's loss lse - z[target]; the backward writes (exp(z - lse) - onehot) scale.  A target outside
// [0, V) is ignored: zero loss and zero gradient.
__device__ __forceinline__ void lse_merge(float& m, float& s, float m2, float s2) {
  const float mm = fmaxf(m, m2);
  if (mm == -INFINITY) return;  // both empty
  s = s * __expf(m - mm) + s2 * __expf(m2 - mm);
  m = mm;
}

__global__ void __launch_bounds__(256) ce_fwd_rows(const float* __restrict__ logits,
                                                   const int32_t* __restrict__ tg, int V,
                                                   float* __restrict__ lse_out, float* __restrict__ row_loss) {
  __shared__ float sm_m[4], sm_s[4];
  const float* z = logits + (int64_t)blockIdx.x * V;
  float m = -INFINITY, s = 0.f;
  if ((V & 3) == 0) {
    const f32x4* z4 = reinterpret_cast<const f32x4*>(z);
    for (int j = threadIdx.x; j < V / 4; j += 256) {
      const f32x4 v = z4[j];
      const float mm = fmaxf(m, fmaxf(fmaxf(v[0], v[1]), fmaxf(v[2], v[3])));
      s = s * __expf(m - mm) + (__expf(v[0] - mm) + __expf(v[1] - mm)) + (__expf(v[2] - mm) + __expf(v[3] - mm));
      m = mm;
    }
  } else {
    for (int j = threadIdx.x; j < V; j += 256) lse_merge(m, s, z[j], 1.f);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float m2 = __shfl_xor(m, o, WAVE), s2 = __shfl_xor(s, o, WAVE);
    lse_merge(m, s, m2, s2);
  }
  if (threadIdx.x % WAVE == 0) {
    sm_m[threadIdx.x / WAVE] = m;
    sm_s[threadIdx.x / WAVE] = s;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    float M = sm_m[0], S = sm_s[0];
    for (int w = 1; w < 4; ++w) lse_merge(M, S, sm_m[w], sm_s[w]);
    const float l = M + __logf(S);
    lse_out[blockIdx.x] = l;
    const int t = tg[blockIdx.x];
    row_loss[blockIdx.x] = (t >= 0 && t < V) ? l - z[t] : 0.f;
  }
}

template <typename T>
__global__ void __launch_bounds__(256) ce_bwd_rows(const float* __restrict__ logits,
                                                   const int32_t* __restrict__ tg,
                                                   const float* __restrict__ lse, int V, float scale,
                                                   T* __restrict__ dlog) {
  const int64_t base = (int64_t)blockIdx.x * V;
  const int t = tg[blockIdx.x];
  const bool valid = t >= 0 && t < V;
  const float l = lse[blockIdx.x];
  const float sc = valid ? scale : 0.f;
  if ((V & 3) == 0) {
    const f32x4* z4 = reinterpret_cast<const f32x4*>(logits + base);
    for (int j = threadIdx.x; j < V / 4; j += 256) {
      const f32x4 v = z4[j];
      float p[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) p[q] = __expf(v[q] - l) * sc - (4 * j + q == t ? sc : 0.f);
      if constexpr (sizeof(T) == 2) {
        bf16x4 o;
#pragma unroll
        for (int q = 0; q < 4; ++q) o[q] = (bf16)p[q];
        *reinterpret_cast<bf16x4*>(dlog + base + 4 * j) = o;
      } else {
        *reinterpret_cast<f32x4*>(dlog + base + 4 * j) = f32x4{p[0], p[1], p[2], p[3]};
      }
    }
  } else {
    for (int j = threadIdx.x; j < V; j += 256)
      dlog[base + j] = from_f32<T>(__expf(logits[base + j] - l) * sc - (j == t ? sc : 0.f));
  }
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
static void gather_t(const int32_t* tok, const void* E, void* x0, int rows, int d, int vocab,
                     hipStream_t st) {
  if (rows <= 0) return;
  if (d % (16 / (int)sizeof(T)) == 0 && ((uintptr_t)E | (uintptr_t)x0) % 16 == 0) {
    embed_gather_vec<T><<<(unsigned)cdiv(rows, 4), 256, 0, st>>>(tok, (const T*)E, (T*)x0, rows, d, vocab);
    return;
  }
  embed_gather<T><<<rows, 256, 0, st>>>(tok, (const T*)E, (T*)x0, d, vocab);
}
void launch_embed_gather(bool bf, const int32_t* tok, const void* table, void* x0, int rows, int d,
                         int vocab, hipStream_t st) {
  DISPATCH(bf, gather_t, tok, table, x0, rows, d, vocab, st);
}

template <typename T>
static void rmsf_t(const void* x, const void* g, void* y, float* r, int rows, int d, float eps,
                   hipStream_t st) {
  const unsigned nv = (unsigned)cdiv(rows, RMS_ROWS_VEC);
  const uintptr_t align = (uintptr_t)x | (uintptr_t)g | (uintptr_t)y;
#define RF(V, NI)                                                                                   \
  if (align % (V * sizeof(T)) == 0) {                                                               \
    rmsnorm_fwd_vec<T, V, NI><<<nv, 256, 0, st>>>((const T*)x, (const T*)g, (T*)y, r, rows, eps);   \
    return;                                                                                         \
  }
  // the row widths of the vectorised backward, plus 4096; any other width, or rows not aligned to
  // the vector, take the block-per-row kernel
  constexpr bool B = sizeof(T) == 2;
  switch (d) {
    case 128: RF(2, 1) break;
    case 256: RF(4, 1) break;
    case 512: if (B) { RF(8, 1) } else { RF(4, 2) } break;
    case 768: RF(4, 3) break;
    case 1024: if (B) { RF(8, 2) } else { RF(4, 4) } break;
    case 1536: if (B) { RF(8, 3) } else { RF(4, 6) } break;
    case 2048: if (B) { RF(8, 4) } else { RF(4, 8) } break;
    case 4096: if (B) { RF(8, 8) } else { RF(4, 16) } break;
    default: break;
  }
#undef RF
  rmsnorm_fwd<T><<<rows, 256, 0, st>>>((const T*)x, (const T*)g, (T*)y, r, d, eps);
}
void launch_rmsnorm_fwd(bool bf, const void* x, const void* gamma, void* y, float* rstd, int rows,
                        int d, float eps, hipStream_t st) {
  DISPATCH(bf, rmsf_t, x, gamma, y, rstd, rows, d, eps, st);
}

template <typename T>
static int rmsb_t(const void* dn, const void* x, const float* r, const void* g, const void* res,
                  void* dx, float* part, int rows, int d, hipStream_t st) {
  const unsigned nv = (unsigned)cdiv(rows, RMS_ROWS_VEC);
  // caller-owned rows (the incoming gradient, dx) may be less aligned than the vector width
  const uintptr_t align = (uintptr_t)dn | (uintptr_t)x | (uintptr_t)g | (uintptr_t)res | (uintptr_t)dx;
#define RB(V, NI)                                                                                    \
  if (align % (V * sizeof(T)) == 0) {                                                                \
    rmsnorm_bwd_vec<T, V, NI><<<nv, 256, 0, st>>>((const T*)dn, (const T*)x, r, (const T*)g,          \
                                                  (const T*)res, (T*)dx, part, rows);                 \
    return (int)nv;                                                                                  \
  }
#define RS(V, NI)                                                                                    \
  if (align % (V * sizeof(T)) == 0) {                                                                \
    rmsnorm_bwd_slice<T, V, NI><<<nv, 256, 0, st>>>((const T*)dn, (const T*)x, r, (const T*)g,        \
                                                    (const T*)res, (T*)dx, part, rows);               \
    return (int)nv;                                                                                  \
  }
  // 16-byte vectors where d allows (8 bf16 or 4 fp32 elements per lane), else 8 or 4 bytes; any
  // other width, or rows not aligned to the vector, take the block-per-chunk kernel below
  constexpr bool B = sizeof(T) == 2;
  switch (d) {
    case 128: RB(2, 1) break;
    case 256: RB(4, 1) break;
    case 512: if (B) { RB(8, 1) } else { RB(4, 2) } break;
    case 768: RB(4, 3) break;
    case 1024: if (B) { RB(8, 2) } else { RB(4, 4) } break;
    case 1536: if (B) { RB(8, 3) } else { RB(4, 6) } break;
    case 2048: if (B) { RS(8, 1) } else { RS(4, 2) } break;
    case 3072: if (B) { RS(4, 3) } else { RS(4, 3) } break;
    case 4096: if (B) { RS(8, 2) } else { RS(4, 4) } break;
    default: break;
  }
#undef RB
#undef RS
  const unsigned nb = (unsigned)cdiv(rows, RMS_CHUNK);
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

void launch_colsum_partials(float* partial, int nchunks, int d, float* out, bool accumulate,
                            hipStream_t st) {
  const unsigned cb = (unsigned)cdiv(d, 256);
  if (nchunks <= 32) {
    colsum_rows<<<dim3(cb, 1), 256, 0, st>>>(partial, nchunks, d, nchunks, out, accumulate ? 1 : 0);
    return;
  }
  constexpr int G = 16;  // rows per first-level group; the group sums go after the partial rows
  const int n1 = cdiv(nchunks, G);
  float* tmp = partial + (int64_t)nchunks * d;
  colsum_rows<<<dim3(cb, (unsigned)n1), 256, 0, st>>>(partial, nchunks, d, G, tmp, 0);
  colsum_rows<<<dim3(cb, 1), 256, 0, st>>>(tmp, n1, d, n1, out, accumulate ? 1 : 0);
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
int64_t token_sort_ws_elems(int n) { return 2 * (int64_t)n + (int64_t)RADIX_DIG * cdiv(n, RADIX_CHUNK); }
void launch_token_sort(const int32_t* tok, int n, int vocab, int32_t* ws, uint32_t* sorted_tok,
                       uint32_t* sorted_pos, hipStream_t st) {
  if (n <= 0) return;
  const int nchunk = (int)cdiv(n, RADIX_CHUNK);
  uint32_t* tk = reinterpret_cast<uint32_t*>(ws);  // the ping-pong partner of (sorted_tok, sorted_pos)
  uint32_t* tv = tk + n;
  int32_t* hist = ws + 2 * (int64_t)n;
  // passes 0 and 2 write the outputs, pass 1 the partner: the last pass ends in sorted_tok / sorted_pos
  uint32_t* ok[RADIX_PASSES] = {sorted_tok, tk, sorted_tok};
  uint32_t* ov[RADIX_PASSES] = {sorted_pos, tv, sorted_pos};
  for (int p = 0; p < RADIX_PASSES; ++p) {
    const int32_t* t0 = p == 0 ? tok : nullptr;
    const uint32_t* ik = p == 0 ? nullptr : ok[p - 1];
    const uint32_t* iv = p == 0 ? nullptr : ov[p - 1];
    radix_count<<<(unsigned)nchunk, 64, 0, st>>>(t0, ik, n, vocab, p * RADIX_BITS, nchunk, hist);
    radix_scan<<<1, 1024, 0, st>>>(hist, RADIX_DIG * nchunk);
    radix_scatter<<<(unsigned)nchunk, 64, 0, st>>>(t0, ik, iv, n, vocab, p * RADIX_BITS, nchunk, hist, ok[p], ov[p]);
  }
}
void launch_token_runs(const uint32_t* sorted_tok, int n, int vocab, int32_t* row_start, int32_t* ids,
                       int32_t* counts, int32_t* n_unique, hipStream_t st) {
  token_row_start<<<(unsigned)cdiv(vocab + 1, 256), 256, 0, st>>>(sorted_tok, n, vocab, row_start);
  if (ids) token_compact<<<1, 1024, 0, st>>>(row_start, vocab, ids, counts, n_unique);
}
void launch_token_compact(const int32_t* row_start, int vocab, int32_t* ids, int32_t* counts, int32_t* n_unique,
                          hipStream_t st) {
  token_compact<<<1, 1024, 0, st>>>(row_start, vocab, ids, counts, n_unique);
}
template <typename T>
static void scat_t(const void* dx0, const uint32_t* sorted_pos, const int32_t* rs, int V, int d,
                   float* de, bool acc, hipStream_t st) {
  embed_scatter<T><<<V, 256, 0, st>>>((const T*)dx0, sorted_pos, rs, d, de, acc ? 1 : 0);
}
void launch_embed_scatter(bool bf, const void* dx0, const uint32_t* sorted_pos,
                          const int32_t* row_start, int vocab, int d, float* de, bool accumulate,
                          hipStream_t st) {
  DISPATCH(bf, scat_t, dx0, sorted_pos, row_start, vocab, d, de, accumulate, st);
}

void launch_ce_fwd(const float* logits, const int32_t* targets, int rows, int vocab, float* lse,
                   float* row_loss, hipStream_t st) {
  if (rows > 0) ce_fwd_rows<<<rows, 256, 0, st>>>(logits, targets, vocab, lse, row_loss);
}
template <typename T>
static void ce_bwd_t(const float* logits, const int32_t* tg, const float* lse, int rows, int V, float scale,
                     void* dl, hipStream_t st) {
  if (rows > 0) ce_bwd_rows<T><<<rows, 256, 0, st>>>(logits, tg, lse, V, scale, (T*)dl);
}
void launch_ce_bwd(bool bf, const float* logits, const int32_t* targets, const float* lse, int rows, int vocab,
                   float scale, void* dlogits, hipStream_t st) {
  DISPATCH(bf, ce_bwd_t, logits, targets, lse, rows, vocab, scale, dlogits, st);
}
void launch_mean(const float* v, int n, float* out, hipStream_t st) {
  mean_kernel<<<1, 1024, 0, st>>>(v, n, out);
}
