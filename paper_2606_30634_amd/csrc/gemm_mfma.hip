// bf16 GEMM on gfx950 matrix cores: C[m, n] (+)= sum_k A(m, k) B(n, k), fp32 accumulation.
//
// v_mfma_f32_32x32x16_bf16: lane l supplies row (l mod 32) of A and of B with the 8 consecutive k
// values 8*(l/32)..+7, and receives C rows 8*(i/4) + 4*(l/32) + (i mod 4), column l mod 32 in
// accumulator i.  Both operands must therefore sit in LDS as [row][k], k contiguous.
//   - an operand whose global layout is k-contiguous (x W^T's x and W, dy W's dy) is copied in
//     16-byte chunks;
//   - an operand whose global layout is row-contiguous (W in dy W, both operands of dy^T x) is
//     read 4 rows x 8 k per thread with 8-byte coalesced loads and transposed in registers.
// Block tile BM x BN x 64, waves WM x WN each, two LDS stages: the next k-slice is fetched into
// registers while the current one feeds the MFMAs, then written to the other stage; one barrier per
// k-slice.  Rows are padded by 16 bytes so the 16-byte fragment reads of 32 rows spread over banks.
// Block order is remapped so that consecutive tiles of one output row band land on one XCD (one L2).
#include "common.h"
#include "kernels.h"
#include <algorithm>

namespace {

constexpr int BK = 64;
constexpr int PADK = BK + 8;  // LDS row pitch in elements

__device__ __forceinline__ uint32_t lo_pair(uint32_t x, uint32_t y) { return (x & 0xffffu) | (y << 16); }
__device__ __forceinline__ uint32_t hi_pair(uint32_t x, uint32_t y) { return (x >> 16) | (y & 0xffff0000u); }

template <int ROWS, int NT, bool KMAJ>
struct TileLoader;

// k-contiguous operand: chunks of 8 consecutive k of one row (16-byte loads and stores)
template <int ROWS, int NT>
struct TileLoader<ROWS, NT, true> {
  static constexpr int CHUNKS = ROWS * BK / 8;
  static constexpr int PER = CHUNKS / NT;
  static_assert(CHUNKS % NT == 0, "tile does not split evenly over the threads");
  uint4 r[PER];

  __device__ __forceinline__ void load(const bf16* __restrict__ G, int ld, int row0, int nrows, int k0,
                                       int K) {
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int c = threadIdx.x + p * NT;
      const int gr = row0 + c / (BK / 8), gk = k0 + (c % (BK / 8)) * 8;
      r[p] = (gr < nrows && gk < K) ? *reinterpret_cast<const uint4*>(G + (int64_t)gr * ld + gk)
                                    : make_uint4(0u, 0u, 0u, 0u);
    }
  }
  __device__ __forceinline__ void store(bf16* __restrict__ S) const {
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int c = threadIdx.x + p * NT;
      *reinterpret_cast<uint4*>(S + (c / (BK / 8)) * PADK + (c % (BK / 8)) * 8) = r[p];
    }
  }
};

// row-contiguous operand: chunks of 4 rows x 8 k; eight 8-byte loads (one per k, lanes along rows)
// are transposed in registers into four 16-byte rows of 8 k
template <int ROWS, int NT>
struct TileLoader<ROWS, NT, false> {
  static constexpr int CHUNKS = ROWS * BK / 32;
  static constexpr int PER = CHUNKS / NT;
  static_assert(CHUNKS % NT == 0, "tile does not split evenly over the threads");
  uint2 r[PER][8];  // r[p][j] = rows 0..3 of the chunk at its k offset j

  __device__ __forceinline__ void load(const bf16* __restrict__ G, int ld, int row0, int nrows, int k0,
                                       int K) {
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int c = threadIdx.x + p * NT;
      const int gr = row0 + (c % (ROWS / 4)) * 4, kb = k0 + (c / (ROWS / 4)) * 8;
#pragma unroll
      for (int j = 0; j < 8; ++j)  // nrows is a multiple of 4: the 4 rows are in bounds together
        r[p][j] = (gr < nrows && kb + j < K) ? *reinterpret_cast<const uint2*>(G + (int64_t)(kb + j) * ld + gr)
                                             : make_uint2(0u, 0u);
    }
  }
  __device__ __forceinline__ void store(bf16* __restrict__ S) const {
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int c = threadIdx.x + p * NT;
      bf16* base = S + ((c % (ROWS / 4)) * 4) * PADK + (c / (ROWS / 4)) * 8;
      uint4 o0, o1, o2, o3;
      o0.x = lo_pair(r[p][0].x, r[p][1].x); o0.y = lo_pair(r[p][2].x, r[p][3].x);
      o0.z = lo_pair(r[p][4].x, r[p][5].x); o0.w = lo_pair(r[p][6].x, r[p][7].x);
      o1.x = hi_pair(r[p][0].x, r[p][1].x); o1.y = hi_pair(r[p][2].x, r[p][3].x);
      o1.z = hi_pair(r[p][4].x, r[p][5].x); o1.w = hi_pair(r[p][6].x, r[p][7].x);
      o2.x = lo_pair(r[p][0].y, r[p][1].y); o2.y = lo_pair(r[p][2].y, r[p][3].y);
      o2.z = lo_pair(r[p][4].y, r[p][5].y); o2.w = lo_pair(r[p][6].y, r[p][7].y);
      o3.x = hi_pair(r[p][0].y, r[p][1].y); o3.y = hi_pair(r[p][2].y, r[p][3].y);
      o3.z = hi_pair(r[p][4].y, r[p][5].y); o3.w = hi_pair(r[p][6].y, r[p][7].y);
      *reinterpret_cast<uint4*>(base) = o0;
      *reinterpret_cast<uint4*>(base + PADK) = o1;
      *reinterpret_cast<uint4*>(base + 2 * PADK) = o2;
      *reinterpret_cast<uint4*>(base + 3 * PADK) = o3;
    }
  }
};

template <int BM, int BN, int WM, int WN, bool AK, bool BKM, typename OutT>
__global__ void __launch_bounds__((BM / WM) * (BN / WN) * 64)
gemm_mfma_kernel(GemmArgs g) {
  constexpr int WAVES_N = BN / WN;
  constexpr int NT = (BM / WM) * (BN / WN) * 64;
  constexpr int FM = WM / 32, FN = WN / 32;
  extern __shared__ __align__(16) unsigned char smem[];
  bf16* As = reinterpret_cast<bf16*>(smem);                 // [2][BM][PADK]
  bf16* Bs = As + 2 * BM * PADK;                            // [2][BN][PADK]

  // XCD-aware tile order: hardware places block b on XCD b mod 8; give each XCD a contiguous run
  // of tiles (in row-band order) so the tiles sharing A rows share that XCD's L2.
  const int tiles_n = (g.N + BN - 1) / BN;
  const int tiles_m = (g.M + BM - 1) / BM;
  const int nblk = tiles_m * tiles_n;
  int b = blockIdx.x;
  if ((nblk & 7) == 0) b = (b & 7) * (nblk >> 3) + (b >> 3);
  const int tm = b / tiles_n, tn = b % tiles_n;
  const int m0 = tm * BM, n0 = tn * BN;

  const int wave = threadIdx.x / 64, lane = threadIdx.x % 64;
  const int wm0 = (wave / WAVES_N) * WM, wn0 = (wave % WAVES_N) * WN;

  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  TileLoader<BM, NT, AK> la;
  TileLoader<BN, NT, BKM> lb;
  const bf16* A = (const bf16*)g.A;
  const bf16* B = (const bf16*)g.B;
  // split-K: this block covers k in [kbeg, kend); kbeg is a multiple of BK
  int kbeg = 0, kend = g.K;
  if (g.ksplit > 1) {
    const int chunk = ((g.K + g.ksplit - 1) / g.ksplit + BK - 1) / BK * BK;
    kbeg = blockIdx.y * chunk;
    kend = min(g.K, kbeg + chunk);
  }
  const int nk = kend > kbeg ? (kend - kbeg + BK - 1) / BK : 0;
  la.load(A, g.lda, m0, g.M, kbeg, kend);
  lb.load(B, g.ldb, n0, g.N, kbeg, kend);
  la.store(As);
  lb.store(Bs);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) {
      la.load(A, g.lda, m0, g.M, kbeg + (kt + 1) * BK, kend);
      lb.load(B, g.ldb, n0, g.N, kbeg + (kt + 1) * BK, kend);
    }
    const bf16* as = As + cur * BM * PADK;
    const bf16* bs = Bs + cur * BN * PADK;
#pragma unroll
    for (int kk = 0; kk < BK; kk += 16) {
      bf16x8 af[FM], bfr[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i)
        af[i] = *reinterpret_cast<const bf16x8*>(as + (wm0 + i * 32 + lane % 32) * PADK + kk + 8 * (lane / 32));
#pragma unroll
      for (int j = 0; j < FN; ++j)
        bfr[j] = *reinterpret_cast<const bf16x8*>(bs + (wn0 + j * 32 + lane % 32) * PADK + kk + 8 * (lane / 32));
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < nk) {
      la.store(As + (cur ^ 1) * BM * PADK);
      lb.store(Bs + (cur ^ 1) * BN * PADK);
    }
    __syncthreads();
  }

  if (g.ksplit > 1) {  // partial tile of this split: plain fp32 into the workspace
    float* W = g.ws + (int64_t)blockIdx.y * g.M * g.N;
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        const int col = n0 + wn0 + j * 32 + lane % 32;
        if (col >= g.N) continue;
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int row = m0 + wm0 + i * 32 + 8 * (e / 4) + 4 * (lane / 32) + (e % 4);
          if (row < g.M) W[(int64_t)row * g.N + col] = acc[i][j][e];
        }
      }
    return;
  }
  OutT* C = (OutT*)g.C;
  const bf16* R = (const bf16*)g.resid;
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int col = n0 + wn0 + j * 32 + lane % 32;
      if (col >= g.N) continue;
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int row = m0 + wm0 + i * 32 + 8 * (e / 4) + 4 * (lane / 32) + (e % 4);
        if (row >= g.M) continue;
        const int64_t o = (int64_t)row * g.ldc + col;
        float v = acc[i][j][e];
        if (sizeof(OutT) == 4 && g.beta != 0.f) v += g.beta * to_f32(C[o]);
        if (R) v += (float)R[o];
        C[o] = from_f32<OutT>(v);
      }
    }
}

// C = beta C + sum over splits of the partial tiles, in split order (fp32 output, ldc == N)
__global__ void __launch_bounds__(256) splitk_reduce(const float* __restrict__ ws, int splits, int64_t mn,
                                                     float* __restrict__ C, float beta) {
  const int64_t i = 4 * ((int64_t)blockIdx.x * blockDim.x + threadIdx.x);
  if (i >= mn) return;
  if (i + 3 < mn) {
    float4 acc = *reinterpret_cast<const float4*>(ws + i);
    for (int s = 1; s < splits; ++s) {
      const float4 v = *reinterpret_cast<const float4*>(ws + (int64_t)s * mn + i);
      acc.x += v.x; acc.y += v.y; acc.z += v.z; acc.w += v.w;
    }
    if (beta != 0.f) {
      const float4 c = *reinterpret_cast<const float4*>(C + i);
      acc.x += beta * c.x; acc.y += beta * c.y; acc.z += beta * c.z; acc.w += beta * c.w;
    }
    *reinterpret_cast<float4*>(C + i) = acc;
  } else {
    for (int64_t k = i; k < mn; ++k) {
      float acc = 0.f;
      for (int s = 0; s < splits; ++s) acc += ws[(int64_t)s * mn + k];
      C[k] = beta != 0.f ? acc + beta * C[k] : acc;
    }
  }
}

template <int BM, int BN, int WM, int WN, typename OutT>
void launch_cfg(const GemmArgs& g, hipStream_t st) {
  constexpr int NT = (BM / WM) * (BN / WN) * 64;
  const size_t lds = (size_t)2 * (BM + BN) * PADK * sizeof(bf16);
  const int nblk = (int)(cdiv(g.M, BM) * cdiv(g.N, BN));
#define L(AK, BKM)                                                                                 \
  do {                                                                                             \
    static bool attr_set = false;                                                                  \
    if (!attr_set) {                                                                               \
      (void)hipFuncSetAttribute((const void*)gemm_mfma_kernel<BM, BN, WM, WN, AK, BKM, OutT>,      \
                                hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);             \
      attr_set = true;                                                                             \
    }                                                                                              \
    gemm_mfma_kernel<BM, BN, WM, WN, AK, BKM, OutT><<<dim3(nblk, g.ksplit), NT, lds, st>>>(g);      \
  } while (0)
  if (g.a_kmajor && g.b_kmajor) L(true, true);
  else if (g.a_kmajor) L(true, false);
  else if (g.b_kmajor) L(false, true);
  else L(false, false);
#undef L
}

}  // namespace

bool gemm_mfma_try(const GemmArgs& g0, hipStream_t st) {
  // vector-load alignment: 8 elements along every contiguous dimension, rows in groups of 4
  if (g0.K % 8 || g0.M % 8 || g0.N % 8 || g0.lda % 8 || g0.ldb % 8) return false;
  if ((uintptr_t)g0.A % 16 || (uintptr_t)g0.B % 16) return false;
  GemmArgs g = g0;
  g.ksplit = 1;
  const int64_t tiles = cdiv(g.M, 128) * cdiv(g.N, 128);
  const int64_t mn = (int64_t)g.M * g.N;
  if (g.out_f32 && g.ws && g.ldc == g.N && tiles < 512 && g.K >= 2048) {
    int s = (int)std::min<int64_t>(8, cdiv(512, tiles));
    while (s > 1 && (s * mn > g.ws_elems || g.K / s < 512)) --s;
    g.ksplit = s;
  }
  if (g.out_f32) launch_cfg<128, 128, 64, 64, float>(g, st);
  else launch_cfg<128, 128, 64, 64, bf16>(g, st);
  if (g.ksplit > 1)
    splitk_reduce<<<(unsigned)cdiv(cdiv(mn, 4), 256), 256, 0, st>>>(g.ws, g.ksplit, mn, (float*)g.C, g.beta);
  return true;
}
