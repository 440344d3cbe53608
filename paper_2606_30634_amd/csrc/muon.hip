// Delayed Muon (Alg. 2 of §4) on the weight matrices of the stage's decoder blocks: the momentum
// update with per-matrix Frobenius norms, the normalised copy in wide orientation (rows <= cols)
// that starts Newton-Schulz, the bf16 hi/lo operand form of an fp32 iterate, and the step that
// applies the orthogonalised update (standard, or the Error-Feedback form of §3.2).  The
// Newton-Schulz products themselves are batched GEMMs launched by the stage.
//
// The iterate X is never rounded to bf16 alone.  That adds noise of relative size 2^-9 in every
// direction, and the iteration multiplies the directions of small singular value by up to
// a = 3.4445 per step: on the low-rank momenta of training that moves O by several percent.  X is
// held in fp32, or as a pair hi + lo of bf16 matrices (hi = bf16(X), lo = bf16(X - hi), X to
// about 2^-17 relative), and the product P X uses the pair.  The Gram matrix A = hi hi^T and
// P = b A + c A A enter as single bf16 matrices: rounding them perturbs X multiplicatively, which
// the small singular directions do not amplify, and A from hi alone differs from X X^T by about
// as much as A's own bf16 rounding does.  On shapes of whole 128 x 128 tiles the
// bf16 stage carries the pair from one step to the next (the product's epilogue forms the next
// pair); other shapes keep X in fp32 and re-split it before each step.
//
// Per matrix W [rows, cols] with delayed gradient g (clipped by c):
//   M <- mu M + (1 - mu) c g
//   X_0 = M / (||M||_F + 1e-7), transposed when rows > cols
//   X_{j+1} = a X_j + (b A + c' A A) X_j, A = X_j X_j^T        (the GEMMs, ns_steps times)
//   u = lr (s O + wd W_t),  O = the last X (transposed back),  s = rms sqrt(max(rows, cols))
//   W_{t+1} = W_t - u, or W_t - (1 + lam) u + lam u_prev;  u_prev <- u;  compute copy of W_{t+1}
// Every reduction has a fixed order (per-chunk partial sums in fp64, summed in chunk order).
#include "common.h"
#include "kernels.h"
#include <cstdio>
#include <cstdlib>

namespace {

constexpr int MU_THREADS = 256;
constexpr int TILE = 64;

// matrix of a block: the last table entry whose first block (first tile) is at or before b
__device__ __forceinline__ int find_mat(const MuonMat* __restrict__ mats, int nmat, int b, bool by_tile) {
  int i = 0;
  while (i + 1 < nmat && (by_tile ? mats[i + 1].tile0 : mats[i + 1].blk0) <= b) ++i;
  return i;
}

// M <- mu M + (1 - mu) c g over MUON_CHUNK elements of one matrix, and the chunk's sum of squares
// of the new M.  A non-finite gradient norm (flag) leaves M as it is.
__global__ void __launch_bounds__(MU_THREADS) muon_momentum(const MuonMat* __restrict__ mats, int nmat,
                                                            const float* __restrict__ g, float* __restrict__ M,
                                                            const float* __restrict__ clip,
                                                            const int* __restrict__ flag, float mu,
                                                            double* __restrict__ partial) {
  __shared__ double sm[16];
  const int i = find_mat(mats, nmat, blockIdx.x, false);
  const MuonMat mm = mats[i];
  const int64_t n = (int64_t)mm.rows * mm.cols;
  const int64_t e0 = (int64_t)(blockIdx.x - mm.blk0) * MUON_CHUNK;
  const int64_t e1 = e0 + MUON_CHUNK < n ? e0 + MUON_CHUNK : n;
  const bool skip = flag && flag[0] != 0;
  const float c = clip ? clip[0] : 1.0f, omm = 1.0f - mu;
  float* Mp = M + mm.off;
  const float* gp = g + mm.off;
  double acc = 0.0;
  for (int64_t e = e0 + 4 * threadIdx.x; e < e1; e += 4 * MU_THREADS) {  // n is a multiple of 4
    f32x4 m = *reinterpret_cast<const f32x4*>(Mp + e);
    if (!skip) {
      const f32x4 gg = *reinterpret_cast<const f32x4*>(gp + e);
#pragma unroll
      for (int q = 0; q < 4; ++q) m[q] = mu * m[q] + omm * (c * gg[q]);
      *reinterpret_cast<f32x4*>(Mp + e) = m;
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) acc += (double)m[q] * m[q];
  }
  acc = block_sum<double>(acc, sm);
  if (threadIdx.x == 0) partial[blockIdx.x] = acc;
}

// norm[i] = sqrt of the sum of matrix i's chunk partials, in chunk order
__global__ void __launch_bounds__(MU_THREADS) muon_norms(const MuonMat* __restrict__ mats, int nmat, int nblk,
                                                         const double* __restrict__ partial,
                                                         float* __restrict__ norm) {
  __shared__ double sm[16];
  const int i = blockIdx.x;
  const int b0 = mats[i].blk0, b1 = i + 1 < nmat ? mats[i + 1].blk0 : nblk;
  double acc = 0.0;
  for (int b = b0 + threadIdx.x; b < b1; b += MU_THREADS) acc += partial[b];
  acc = block_sum<double>(acc, sm);
  if (threadIdx.x == 0) norm[i] = (float)sqrt(acc);
}

// X_0 of one 64 x 64 tile of a matrix: M / (||M|| + 1e-7), transposed through LDS when the
// workspace holds the transpose.
__global__ void __launch_bounds__(MU_THREADS) muon_prep(const MuonMat* __restrict__ mats, int nmat,
                                                        const float* __restrict__ M, const float* __restrict__ norm) {
  __shared__ float tile[TILE][TILE + 1];
  const int i = find_mat(mats, nmat, blockIdx.x, true);
  const MuonMat mm = mats[i];
  const int tcols = (mm.cols + TILE - 1) / TILE;
  const int t = blockIdx.x - mm.tile0;
  const int r0 = (t / tcols) * TILE, c0 = (t % tcols) * TILE;
  const float inv = 1.0f / (norm[i] + 1e-7f);
  const float* Mp = M + mm.off;
  float* X = mm.x[0];
  const int tx = threadIdx.x % TILE, ty = threadIdx.x / TILE;  // 64 x 4
  for (int k = ty; k < TILE; k += MU_THREADS / TILE) {
    const int r = r0 + k, c = c0 + tx;
    tile[k][tx] = (r < mm.rows && c < mm.cols) ? Mp[(int64_t)r * mm.cols + c] * inv : 0.f;
  }
  __syncthreads();
  if (!mm.trans) {
    for (int k = ty; k < TILE; k += MU_THREADS / TILE) {
      const int r = r0 + k, c = c0 + tx;
      if (r < mm.rows && c < mm.cols) X[(int64_t)r * mm.cols + c] = tile[k][tx];
    }
  } else {  // X is [cols][rows]: row c of X holds column c of M
    for (int k = ty; k < TILE; k += MU_THREADS / TILE) {
      const int c = c0 + k, r = r0 + tx;
      if (r < mm.rows && c < mm.cols) X[(int64_t)c * mm.rows + r] = tile[tx][k];
    }
  }
}

// The update of one 64 x 64 tile of a matrix from O = x[fin] (transposed back through LDS):
// u = lr (s O + wd W), the standard or Error-Feedback step, u_prev <- u, and the compute copy.
// A non-finite gradient norm (flag) leaves W and u_prev as they are and writes the copy only.
template <typename S>
__global__ void __launch_bounds__(MU_THREADS) muon_apply(const MuonMat* __restrict__ mats, int nmat, int fin,
                                                         float* __restrict__ W, float* __restrict__ up,
                                                         S* __restrict__ shadow, const int* __restrict__ flag,
                                                         float lr, float wd, float rms, int ef, float lam) {
  __shared__ float tile[TILE][TILE + 1];
  const int i = find_mat(mats, nmat, blockIdx.x, true);
  const MuonMat mm = mats[i];
  const int tcols = (mm.cols + TILE - 1) / TILE;
  const int t = blockIdx.x - mm.tile0;
  const int r0 = (t / tcols) * TILE, c0 = (t % tcols) * TILE;
  const float* X = mm.x[fin];
  const int tx = threadIdx.x % TILE, ty = threadIdx.x / TILE;
  if (mm.trans) {  // X is [cols][rows]
    for (int k = ty; k < TILE; k += MU_THREADS / TILE) {
      const int c = c0 + k, r = r0 + tx;
      tile[tx][k] = (r < mm.rows && c < mm.cols) ? X[(int64_t)c * mm.rows + r] : 0.f;
    }
    __syncthreads();
  }
  const bool skip = flag && flag[0] != 0;
  const float s = rms * mm.sqrt_max, onep = 1.0f + lam;
  for (int k = ty; k < TILE; k += MU_THREADS / TILE) {
    const int r = r0 + k, c = c0 + tx;
    if (r >= mm.rows || c >= mm.cols) continue;
    const int64_t e = mm.off + (int64_t)r * mm.cols + c;
    float w = W[e];
    if (!skip) {
      const float o = mm.trans ? tile[k][tx] : X[(int64_t)r * mm.cols + c];
      const float u = lr * (s * o + wd * w);
      w = ef ? w - onep * u + lam * up[e] : w - u;
      W[e] = w;
      if (up) up[e] = u;
    }
    shadow[e] = from_f32<S>(w);
  }
}

// S row r = [hi | lo] of X row r, V consecutive columns per thread
template <int V>
__global__ void __launch_bounds__(MU_THREADS) muon_split(const float* __restrict__ X, bf16* __restrict__ S,
                                                         int64_t rows, int n) {
  const int64_t per_row = n / V;
  const int64_t i = (int64_t)blockIdx.x * MU_THREADS + threadIdx.x;
  if (i >= rows * per_row) return;
  const int64_t r = i / per_row;
  const int c = (int)(i % per_row) * V;
  const float* x = X + r * n + c;
  bf16* s = S + r * 2 * n + c;
  if constexpr (V == 4) {
    const f32x4 v = *reinterpret_cast<const f32x4*>(x);
    bf16x4 hi, lo;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      hi[q] = (bf16)v[q];
      lo[q] = (bf16)(v[q] - (float)hi[q]);
    }
    *reinterpret_cast<bf16x4*>(s) = hi;
    *reinterpret_cast<bf16x4*>(s + n) = lo;
  } else {
    const bf16 hi = (bf16)x[0], lo = (bf16)(x[0] - (float)hi);
    s[0] = hi;
    s[n] = lo;
  }
}

// X row r = hi + lo of S row r = [hi | lo], 4 consecutive columns per thread
__global__ void __launch_bounds__(MU_THREADS) muon_join(const bf16* __restrict__ S, float* __restrict__ X,
                                                        int64_t rows, int n) {
  const int64_t per_row = n / 4;
  const int64_t i = (int64_t)blockIdx.x * MU_THREADS + threadIdx.x;
  if (i >= rows * per_row) return;
  const int64_t r = i / per_row;
  const int c = (int)(i % per_row) * 4;
  const bf16* s = S + r * 2 * n + c;
  const bf16x4 hi = *reinterpret_cast<const bf16x4*>(s);
  const bf16x4 lo = *reinterpret_cast<const bf16x4*>(s + n);
  f32x4 v;
#pragma unroll
  for (int q = 0; q < 4; ++q) v[q] = (float)hi[q] + (float)lo[q];
  *reinterpret_cast<f32x4*>(X + r * n + c) = v;
}

}  // namespace

int64_t muon_chunks(int64_t numel) { return (numel + MUON_CHUNK - 1) / MUON_CHUNK; }
int64_t muon_tiles(int rows, int cols) { return (int64_t)((rows + TILE - 1) / TILE) * ((cols + TILE - 1) / TILE); }

void launch_muon_momentum(const MuonMat* mats, int nmat, int nblk, const float* g, float* M, const float* clip,
                          const int* flag, float mu, double* partial, float* norm, hipStream_t st) {
  muon_momentum<<<nblk, MU_THREADS, 0, st>>>(mats, nmat, g, M, clip, flag, mu, partial);
  muon_norms<<<nmat, MU_THREADS, 0, st>>>(mats, nmat, nblk, partial, norm);
}

void launch_muon_prep(const MuonMat* mats, int nmat, int ntile, const float* M, const float* norm, hipStream_t st) {
  muon_prep<<<ntile, MU_THREADS, 0, st>>>(mats, nmat, M, norm);
}

void launch_muon_split(const float* X, bf16* S, int64_t rows, int n, hipStream_t st) {
  if (rows == 0 || n == 0) return;
  if (n % 4 == 0)
    muon_split<4><<<(unsigned)((rows * (n / 4) + MU_THREADS - 1) / MU_THREADS), MU_THREADS, 0, st>>>(X, S, rows, n);
  else
    muon_split<1><<<(unsigned)((rows * n + MU_THREADS - 1) / MU_THREADS), MU_THREADS, 0, st>>>(X, S, rows, n);
}

void launch_muon_join(const bf16* S, float* X, int64_t rows, int n, hipStream_t st) {
  if (rows == 0 || n == 0) return;
  if (n % 4) {
    fprintf(stderr, "launch_muon_join: n = %d is not a multiple of 4\n", n);
    abort();
  }
  muon_join<<<(unsigned)((rows * (n / 4) + MU_THREADS - 1) / MU_THREADS), MU_THREADS, 0, st>>>(S, X, rows, n);
}

void launch_muon_apply(bool bf, const MuonMat* mats, int nmat, int ntile, int fin, float* W, float* up,
                       void* shadow, const int* flag, float lr, float wd, float rms, bool ef, float lam,
                       hipStream_t st) {
  if (bf)
    muon_apply<bf16><<<ntile, MU_THREADS, 0, st>>>(mats, nmat, fin, W, up, (bf16*)shadow, flag, lr, wd, rms,
                                                         ef ? 1 : 0, lam);
  else
    muon_apply<float><<<ntile, MU_THREADS, 0, st>>>(mats, nmat, fin, W, up, (float*)shadow, flag, lr, wd,
                                                           rms, ef ? 1 : 0, lam);
}
