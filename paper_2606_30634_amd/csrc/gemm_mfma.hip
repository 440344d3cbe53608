// bf16 GEMM on gfx950 matrix cores: C[m, n] (+)= sum_k A(m, k) B(n, k), fp32 accumulation.
//
// v_mfma_f32_32x32x16_bf16: lane l supplies row (l mod 32) of A and of B with the 8 consecutive k
// values 8*(l/32)..+7, and receives C rows 8*(i/4) + 4*(l/32) + (i mod 4), column l mod 32 in
// accumulator i.  Both operands therefore sit in LDS as [row][k], k contiguous.
//   - an operand whose global layout is k-contiguous (x W^T's x and W, dy W's dy) is copied in
//     16-byte chunks;
//   - an operand whose global layout is row-contiguous (W in dy W, both operands of dy^T x) is
//     staged as it sits in memory ([k][row], 16-byte chunks) and its fragments are read with
//     gfx950's transposing LDS read ds_read_b64_tr_b16.
// Block tile BM x BN x 64 over 4 waves of WM x WN, two LDS stages: the next k-slice is fetched into
// registers while the current one feeds the MFMAs, then written to the other stage; one barrier per
// k-slice.  Inside a k-slice the fragments of the next 16-deep step are read from LDS while the
// MFMAs of the current one run.  Rows are padded by 16 bytes so the 16-byte fragment reads of 32
// rows spread over the banks.  Full tiles use loaders without bounds checks.  The epilogue stages
// each wave's tile through LDS, 32 rows at a time, and writes 16-byte rows (residual and beta
// terms read the same way).  Block order is remapped so that consecutive tiles of one output row
// band land on one XCD (one L2).  Deterministic split-K for underfilled fp32-output products.
#include "common.h"
#include "kernels.h"
#include <algorithm>

namespace {

constexpr int BK = 64;
constexpr int PADK = BK + 8;  // LDS row pitch in elements

template <int ROWS, int NT, bool KMAJ, bool CHECK>
struct TileLoader;

// k-contiguous operand: chunks of 8 consecutive k of one row (16-byte loads and stores)
template <int ROWS, int NT, bool CHECK>
struct TileLoader<ROWS, NT, true, CHECK> {
  static constexpr int CHUNKS = ROWS * BK / 8;
  static constexpr int PER = CHUNKS / NT;
  static_assert(CHUNKS % NT == 0, "tile does not split evenly over the threads");
  u32x4 r[PER];

  __device__ __forceinline__ void load(const bf16* __restrict__ G, int ld, int row0, int nrows, int k0,
                                       int K) {
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int c = threadIdx.x + p * NT;
      const int gr = row0 + c / (BK / 8), gk = k0 + (c % (BK / 8)) * 8;
      const bool ok = !CHECK || (gr < nrows && gk < K);
      const u32x4 v = ok ? *reinterpret_cast<const u32x4*>(G + (int64_t)gr * ld + gk) : u32x4{0u, 0u, 0u, 0u};
      r[p] = v;
    }
  }
  __device__ __forceinline__ void store_one(bf16* __restrict__ S, int p) const {
    const int c = threadIdx.x + p * NT;
    *reinterpret_cast<u32x4*>(S + (c / (BK / 8)) * PADK + (c % (BK / 8)) * 8) = r[p];
  }
  __device__ __forceinline__ void store(bf16* __restrict__ S) const {
#pragma unroll
    for (int p = 0; p < PER; ++p) store_one(S, p);
  }
};

// row-contiguous operand: kept as it sits in memory, a [k][row] tile of pitch ROWS + 32 filled
// with 16-byte chunks of 8 rows; its MFMA fragments are read with transposing LDS reads.  One
// such read by half a wave covers 4 k-rows x 32 rows (16 dwords per k-row); a pitch of 16 dwords
// mod 64 puts those four runs on disjoint banks.
template <int ROWS>
constexpr int row_pitch() { return ROWS + 32; }

template <int ROWS, int NT, bool CHECK>
struct TileLoader<ROWS, NT, false, CHECK> {
  static constexpr int CHUNKS = ROWS * BK / 8;
  static constexpr int PER = CHUNKS / NT;
  static constexpr int PR = row_pitch<ROWS>();
  static_assert(CHUNKS % NT == 0, "tile does not split evenly over the threads");
  u32x4 r[PER];

  __device__ __forceinline__ void load(const bf16* __restrict__ G, int ld, int row0, int nrows, int k0,
                                       int K) {
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int c = threadIdx.x + p * NT;
      const int gk = k0 + c / (ROWS / 8), gr = row0 + (c % (ROWS / 8)) * 8;
      const bool ok = !CHECK || (gr < nrows && gk < K);  // nrows is a multiple of 8
      r[p] = ok ? *reinterpret_cast<const u32x4*>(G + (int64_t)gk * ld + gr) : u32x4{0u, 0u, 0u, 0u};
    }
  }
  __device__ __forceinline__ void store_one(bf16* __restrict__ S, int p) const {
    const int c = threadIdx.x + p * NT;
    *reinterpret_cast<u32x4*>(S + (c / (ROWS / 8)) * PR + (c % (ROWS / 8)) * 8) = r[p];
  }
  __device__ __forceinline__ void store(bf16* __restrict__ S) const {
#pragma unroll
    for (int p = 0; p < PER; ++p) store_one(S, p);
  }
};

// LDS elements of one stage of an operand tile
template <int ROWS, bool KMAJ>
constexpr int stage_elems() { return KMAJ ? ROWS * PADK : BK * row_pitch<ROWS>(); }

// MFMA fragment: row r0 + lane mod 32 of the tile, k = k0 + 8 (lane / 32) .. +7
template <int ROWS, bool KMAJ>
__device__ __forceinline__ bf16x8 frag(const bf16* T, int r0, int k0) {
  if constexpr (KMAJ) {
    const int l = threadIdx.x % 64;
    return *reinterpret_cast<const bf16x8*>(T + (r0 + l % 32) * PADK + k0 + 8 * (l / 32));
  } else {
    return frag_tr(T, row_pitch<ROWS>(), r0, k0);
  }
}

template <int BM, int BN, int WM, int WN, bool AK = true, bool BKM = true>
struct Cfg {
  static constexpr int NW = (BM / WM) * (BN / WN);
  static constexpr int NT = NW * 64;
  static constexpr int FM = WM / 32, FN = WN / 32;
  static constexpr int SA = stage_elems<BM, AK>(), SB = stage_elems<BN, BKM>();
  static constexpr size_t main_lds = (size_t)2 * (SA + SB) * sizeof(bf16);
  static constexpr int EP = WN + 4;  // epilogue staging pitch (fp32 elements)
  static constexpr size_t epi_lds = (size_t)NW * 16 * EP * sizeof(float);
  static constexpr size_t lds = main_lds > epi_lds ? main_lds : epi_lds;
};

// Waves per SIMD the tile allows (accumulators and LDS stages): told to the compiler so that it
// schedules for that occupancy instead of trading the fragment prefetch for registers.
template <int BM, int BN>
constexpr int tile_waves_per_simd() { return BM * BN >= 256 * 256 ? 1 : 2; }

// XCD-aware tile order: hardware places block b on XCD b mod 8; give each XCD a contiguous run
// of tiles, walked in groups of GM row tiles (down a group's rows, then to its next column), so
// the blocks resident on one XCD at a time cover a compact patch of C and share their A and B
// slices in that XCD's L2.
template <int BM, int BN>
__device__ __forceinline__ void tile_origin(const GemmArgs& g, int b, int& m0, int& n0) {
  constexpr int GM = 8;
  const int tiles_n = (g.N + BN - 1) / BN;
  const int tiles_m = (g.M + BM - 1) / BM;
  const int nblk = tiles_m * tiles_n;
  if ((nblk & 7) == 0) b = (b & 7) * (nblk >> 3) + (b >> 3);
  const int first_m = (b / (GM * tiles_n)) * GM;
  const int gsz = min(tiles_m - first_m, GM);
  m0 = (first_m + (b % (GM * tiles_n)) % gsz) * BM;
  n0 = ((b % (GM * tiles_n)) / gsz) * BN;
}

// Tile b of a symmetric product (M == N, square tiles): the b-th tile (i, j) with i <= j, counted
// row by row (T (T + 1) / 2 tiles for T tile rows).
template <int BM, int BN>
__device__ __forceinline__ void tri_origin(const GemmArgs& g, int b, int& m0, int& n0) {
  static_assert(BM == BN, "square tiles");
  const int T = g.M / BM;
  int i = 0, first = 0;
  while (i + 1 < T && b >= first + (T - i)) {
    first += T - i;
    ++i;
  }
  m0 = i * BM;
  n0 = (i + b - first) * BN;
}

// Epilogue: per RP-row part (RP = 16 or 8) of each 32-row fragment row of the wave tile, stage
// the fp32 accumulators through the wave's own LDS area and write 16-byte rows: split-K partials
// to the workspace, or C with the beta / residual / SwiGLU-backward / RoPE / delta /
// SwiGLU-forward terms.  A wave reads back only what it wrote, and one wave's LDS operations
// complete in issue order, so no barrier is needed between the parts and the global stores are
// never waited for here.  The staging area (NW x RP x (WN + 4) floats) must be free: every wave
// past its last read of it.
template <int BM, int BN, int WM, int WN, typename OutT, bool CHECK, int RP = 16>
__device__ __forceinline__ void gemm_epilogue(const GemmArgs& g, f32x16 (&acc)[WM / 32][WN / 32],
                                              float* stage, int m0, int n0, int wm0, int wn0) {
  static_assert(RP == 16 || RP == 8, "staging part of 8 or 16 rows");
  constexpr int FM = WM / 32, FN = WN / 32;
  constexpr int EP = WN + 4;  // staging pitch (fp32 elements)
  constexpr int NP = 32 / RP, EPP = 16 / NP;  // parts per fragment row, accumulators per part
  const int wave = threadIdx.x / 64, lane = threadIdx.x % 64;
  float* stg = stage + wave * RP * EP;
  const bool split = g.ksplit > 1;
  float* W = split ? g.ws + (int64_t)blockIdx.y * g.M * g.N : nullptr;
  OutT* C = (OutT*)g.C;
  const bf16* R = (const bf16*)g.resid;
  constexpr int VEC = sizeof(OutT) == 2 ? 8 : 4;  // elements per 16-byte store
  static_for<FM * NP>([&](auto IH) {
    constexpr int i = IH / NP, h = IH % NP;
    // accumulator e of lane l holds fragment row 8 (e / 4) + 4 (l / 32) + e mod 4: rows
    // RP h .. RP h + RP - 1 are e = EPP h .. EPP h + EPP - 1
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int e = EPP * h; e < EPP * h + EPP; ++e)
        stg[(8 * (e / 4) - RP * h + 4 * (lane / 32) + (e % 4)) * EP + j * 32 + lane % 32] = acc[i][j][e];
    asm volatile("" ::: "memory");
    const int rbase = m0 + wm0 + i * 32 + RP * h;
    if (split) {
      for (int c = lane; c < RP * WN / 4; c += 64) {
        const int r = c / (WN / 4), cc = (c % (WN / 4)) * 4;
        const int row = rbase + r, col = n0 + wn0 + cc;
        if (!CHECK || (row < g.M && col < g.N))
          *reinterpret_cast<float4*>(W + (int64_t)row * g.N + col) = *reinterpret_cast<const float4*>(stg + r * EP + cc);
      }
    } else {
      for (int c = lane; c < RP * WN / VEC; c += 64) {
        const int r = c / (WN / VEC), cc = (c % (WN / VEC)) * VEC;
        const int row = rbase + r, col = n0 + wn0 + cc;
        if (CHECK && (row >= g.M || col >= g.N)) continue;  // N is a multiple of 8
        const int64_t o = (int64_t)row * g.ldc + col;
        float v[VEC];
#pragma unroll
        for (int q = 0; q < VEC; ++q) v[q] = stg[r * EP + cc + q];
        if constexpr (sizeof(OutT) == 4) {
          if (g.beta != 0.f) {
            const float4 old = *reinterpret_cast<const float4*>((const float*)C + o);
            v[0] += g.beta * old.x; v[1] += g.beta * old.y; v[2] += g.beta * old.z; v[3] += g.beta * old.w;
          }
          *reinterpret_cast<float4*>((float*)C + o) = make_float4(v[0], v[1], v[2], v[3]);
        } else if (g.epi == 1) {  // SwiGLU backward from dz = v
          const bf16* gu = (const bf16*)g.aux + (int64_t)row * g.ld_aux + col;
          const bf16x8 av = *reinterpret_cast<const bf16x8*>(gu);
          const bf16x8 bv = *reinterpret_cast<const bf16x8*>(gu + g.N);
          bf16x8 da, db;
#pragma unroll
          for (int q = 0; q < 8; ++q) {
            const float a = (float)av[q], bb = (float)bv[q];
            const float sg = 1.0f / (1.0f + __expf(-a));
            da[q] = (bf16)(v[q] * bb * sg * (1.0f + a * (1.0f - sg)));
            db[q] = (bf16)(v[q] * a * sg);
          }
          *reinterpret_cast<bf16x8*>((bf16*)C + o) = da;
          *reinterpret_cast<bf16x8*>((bf16*)C + o + g.N) = db;
        } else if (g.epi == 4) {  // dO, plus delta = rowsum(dO O) over each head's columns
          bf16x8 ov;
#pragma unroll
          for (int q = 0; q < 8; ++q) ov[q] = (bf16)v[q];
          *reinterpret_cast<bf16x8*>((bf16*)C + o) = ov;
          const bf16x8 ob = *reinterpret_cast<const bf16x8*>((const bf16*)g.aux + (int64_t)row * g.ld_aux + col);
          float dot = 0.f;
#pragma unroll
          for (int q = 0; q < 8; ++q) dot += (float)ov[q] * (float)ob[q];
          // the head's delta_hd / 8 chunks sit in consecutive lanes (aligned groups)
          for (int m = 1; m < g.delta_hd / 8; m <<= 1) dot += __shfl_xor(dot, m, 64);
          if (col % g.delta_hd == 0) {
            const int bb = row / g.delta_S, ii = row % g.delta_S, hh = col / g.delta_hd;
            g.delta[((int64_t)bb * (g.N / g.delta_hd) + hh) * g.delta_S + ii] = dot;
          }
        } else if (g.epi == 3) {  // SwiGLU forward: panel column col is gate or up of z column zc
          const int grp = col / 32, zc = (grp / 2) * 32 + col % 32;
          bf16x8 ov;
#pragma unroll
          for (int q = 0; q < 8; ++q) ov[q] = (bf16)v[q];
          bf16* Cb = (bf16*)C + (int64_t)row * g.ldc;
          if ((grp & 1) == 0) {
            *reinterpret_cast<bf16x8*>(Cb + zc) = ov;
            const float* up = stg + r * EP + cc + 32;  // the up values of the same z columns
            bf16x8 zv;
#pragma unroll
            for (int q = 0; q < 8; ++q) zv[q] = (bf16)(v[q] / (1.0f + __expf(-v[q])) * up[q]);
            *reinterpret_cast<bf16x8*>((bf16*)g.out2 + (int64_t)row * g.ld_out2 + zc) = zv;
          } else {
            *reinterpret_cast<bf16x8*>(Cb + g.glu + zc) = ov;
          }
        } else if (g.epi == 2 && col < g.rope_cols) {  // RoPE on the fp32 products
          const int hd = g.rope_hd, hh = hd / 2;
          const int c = col % hd, i0 = c % hh;
          const bool first = c < hh;
          const float* xp = stg + r * EP + (first ? cc + hh : cc - hh);  // partner columns
          const int64_t tb = (int64_t)(row % g.rope_S) * hh + i0;
          bf16x8 ov;
#pragma unroll
          for (int q = 0; q < 8; ++q) {
            const float cs = g.rope_cos[tb + q], sn = g.rope_sin[tb + q];
            ov[q] = (bf16)(first ? v[q] * cs - xp[q] * sn : v[q] * cs + xp[q] * sn);
          }
          *reinterpret_cast<bf16x8*>((bf16*)C + o) = ov;
        } else {
          if (R) {
            const bf16x8 rr = *reinterpret_cast<const bf16x8*>(R + o);
#pragma unroll
            for (int q = 0; q < 8; ++q) v[q] += (float)rr[q];
          }
          bf16x8 ov;
#pragma unroll
          for (int q = 0; q < 8; ++q) ov[q] = (bf16)v[q];
          *reinterpret_cast<bf16x8*>((bf16*)C + o) = ov;
        }
      }
    }
    asm volatile("" ::: "memory");
  });
}

// Epilogue kinds of the direct-to-LDS kernels (compile-time; the numbers of the first five are
// GemmArgs::epi): bf16 output as is, SwiGLU backward, RoPE, SwiGLU forward, attention delta, plus
// a residual row added, alpha (A B) + beta D.
enum { EPI_PLAIN = 0, EPI_SWIGLU_BWD = 1, EPI_ROPE = 2, EPI_SWIGLU_FWD = 3, EPI_DELTA = 4, EPI_RESID = 5,
       EPI_AXPBY = GEMM_EPI_AXPBY, EPI_AXPBY_DUP = GEMM_EPI_AXPBY_DUP, EPI_NS_SPLIT = GEMM_EPI_NS_SPLIT };

// Output chunks leave with non-temporal stores and read-once epilogue operands arrive with
// non-temporal loads: a product streams 10-150 MB of them through the 4 MB L2 of each XCD, which
// would otherwise evict the operand panels that the tiles resident on the XCD share.
template <typename V>
__device__ __forceinline__ void st_nt(void* p, const V& v) {
  static_assert(sizeof(V) == 16, "16-byte chunk");
  u32x4 u;
  __builtin_memcpy(&u, &v, 16);
  __builtin_nontemporal_store(u, reinterpret_cast<u32x4*>(p));
}
template <typename V>
__device__ __forceinline__ V ld_nt(const void* p) {
  static_assert(sizeof(V) == 16, "16-byte chunk");
  const u32x4 u = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
  V v;
  __builtin_memcpy(&v, &u, 16);
  return v;
}

// Global operands of one 16-byte output chunk (8 bf16 columns) that an epilogue reads.
template <int EPI> struct EpiIn { static constexpr bool loads = false; };
template <> struct EpiIn<EPI_RESID> { static constexpr bool loads = true; bf16x8 r; };
template <> struct EpiIn<EPI_AXPBY> { static constexpr bool loads = true; bf16x8 r; };
template <> struct EpiIn<EPI_AXPBY_DUP> { static constexpr bool loads = true; bf16x8 r; };
template <> struct EpiIn<EPI_NS_SPLIT> { static constexpr bool loads = true; bf16x8 a, b; };
template <> struct EpiIn<EPI_SWIGLU_BWD> { static constexpr bool loads = true; bf16x8 a, b; };
template <> struct EpiIn<EPI_DELTA> { static constexpr bool loads = true; f32x4 o0, o1; };
template <> struct EpiIn<EPI_ROPE> { static constexpr bool loads = true; f32x4 c0, c1, s0, s1; };

template <int EPI>
__device__ __forceinline__ void epi_load(EpiIn<EPI>& in, const GemmArgs& g, int row, int col) {
  if constexpr (EPI == EPI_RESID) {
    in.r = ld_nt<bf16x8>((const bf16*)g.resid + (int64_t)row * g.ldc + col);
  } else if constexpr (EPI == EPI_AXPBY) {
    in.r = ld_nt<bf16x8>((const bf16*)g.D + (int64_t)row * g.ldc + col);
  } else if constexpr (EPI == EPI_AXPBY_DUP) {
    in.r = ld_nt<bf16x8>((const bf16*)g.D + (int64_t)row * g.ld_aux + col);
  } else if constexpr (EPI == EPI_NS_SPLIT) {  // hi and lo of the previous x
    const bf16* dp = (const bf16*)g.D + (int64_t)row * g.ldc + col;
    in.a = ld_nt<bf16x8>(dp);
    in.b = ld_nt<bf16x8>(dp + g.N);
  } else if constexpr (EPI == EPI_SWIGLU_BWD) {
    const bf16* gu = (const bf16*)g.aux + (int64_t)row * g.ld_aux + col;
    in.a = ld_nt<bf16x8>(gu);
    in.b = ld_nt<bf16x8>(gu + g.N);
  } else if constexpr (EPI == EPI_DELTA) {
    const float* op = (const float*)g.aux + (int64_t)row * g.ld_aux + col;
    in.o0 = ld_nt<f32x4>(op);
    in.o1 = ld_nt<f32x4>(op + 4);
  } else if constexpr (EPI == EPI_ROPE) {
    if (col < g.rope_cols) {
      const int hh = g.rope_hd / 2, i0 = (col % g.rope_hd) % hh;
      const int64_t tb = (int64_t)(row % g.rope_S) * hh + i0;
      in.c0 = *reinterpret_cast<const f32x4*>(g.rope_cos + tb);
      in.c1 = *reinterpret_cast<const f32x4*>(g.rope_cos + tb + 4);
      in.s0 = *reinterpret_cast<const f32x4*>(g.rope_sin + tb);
      in.s1 = *reinterpret_cast<const f32x4*>(g.rope_sin + tb + 4);
    }
  }
}

__device__ __forceinline__ float sigmoid_fast(float a) {
  return __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(-1.4426950408889634f * a));
}

// Epilogue of the direct-to-LDS kernels (full tiles).  Per RP-row part of each 32-row fragment
// row of the wave tile: the accumulators go through the wave's own LDS staging area and leave as
// 16-byte rows.  The global operands the epilogue kind reads are all requested before the first
// part is written (or one part ahead, where the registers for all of them would not fit), so their
// latency is paid about once per tile instead of once per part.  A wave reads back only what it wrote and
// its LDS operations complete in issue order: no barrier between parts, and the stores are never
// waited for here.  The staging area (waves x RP x (WN + 4) floats) must be free.
template <int BM, int BN, int WM, int WN, typename OutT, int EPI, int RP>
__device__ __forceinline__ void dma_epilogue(const GemmArgs& g, f32x16 (&acc)[WM / 32][WN / 32],
                                             float* stage, int m0, int n0, int wm0, int wn0) {
  static_assert(RP == 16 || RP == 8, "staging part of 8 or 16 rows");
  static_assert(sizeof(OutT) == 2 || EPI == EPI_PLAIN, "fp32 output has no fused epilogue");
  constexpr int FM = WM / 32, FN = WN / 32;
  constexpr int EP = WN + 4;  // staging pitch (fp32 elements)
  constexpr int NP = 32 / RP, EPP = 16 / NP;  // parts per fragment row, accumulators per part
  constexpr int VEC = sizeof(OutT) == 2 ? 8 : 4;  // elements per 16-byte chunk
  constexpr int CPR = WN / VEC;                   // chunks per staged row
  constexpr int CPL = RP * CPR / 64;              // chunks per lane and part
  constexpr int NPART = FM * NP;
  static_assert(CPL * 64 == RP * CPR, "every lane writes the same number of chunks per part");
  // Parts requested ahead of the one being written, within a per-lane register budget for the
  // requested operands (the wider wave tile holds more accumulators): all of them, one, or none.
  constexpr int PART_BYTES = EpiIn<EPI>::loads ? CPL * (int)sizeof(EpiIn<EPI>) : 0;
  constexpr int BUDGET = WN <= 64 ? 256 : 128;
  constexpr int PD = PART_BYTES == 0 ? 0
                     : PART_BYTES * NPART <= BUDGET ? NPART
                     : 2 * PART_BYTES <= BUDGET ? 1 : 0;
  constexpr int RS = PD >= NPART ? NPART : PD + 1;  // ring of requested parts
  const int wave = threadIdx.x / 64, lane = threadIdx.x % 64;
  float* stg = stage + wave * RP * EP;
  const bool split = sizeof(OutT) == 4 && g.ksplit > 1;
  float* W = split ? g.ws + (int64_t)blockIdx.y * g.M * g.N : nullptr;
  // output chunk j of part p of this lane: staged row r, column cc; C row, column
  auto chunk = [&](int p, int j, int& r, int& cc, int& row, int& col) {
    const int c = lane + 64 * j;
    r = c / CPR;
    cc = (c % CPR) * VEC;
    row = m0 + wm0 + (p / NP) * 32 + RP * (p % NP) + r;
    col = n0 + wn0 + cc;
  };
  EpiIn<EPI> in[RS][CPL];
  auto request = [&](auto P) {
    constexpr int p = P;
#pragma unroll
    for (int j = 0; j < CPL; ++j) {
      int r, cc, row, col;
      chunk(p, j, r, cc, row, col);
      epi_load<EPI>(in[p % RS][j], g, row, col);
    }
  };
  if constexpr (PD > 0) static_for<(PD < NPART ? PD : NPART)>(request);
  static_for<NPART>([&](auto P) {
    constexpr int p = P, i = p / NP, h = p % NP;
    if constexpr (EpiIn<EPI>::loads && p + PD < NPART) request(std::integral_constant<int, p + PD>{});
    // accumulator e of lane l holds fragment row 8 (e / 4) + 4 (l / 32) + e mod 4: rows
    // RP h .. RP h + RP - 1 are e = EPP h .. EPP h + EPP - 1
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int e = EPP * h; e < EPP * h + EPP; ++e)
        stg[(8 * (e / 4) - RP * h + 4 * (lane / 32) + (e % 4)) * EP + j * 32 + lane % 32] = acc[i][j][e];
    asm volatile("" ::: "memory");
#pragma unroll
    for (int j = 0; j < CPL; ++j) {
      int r, cc, row, col;
      chunk(p, j, r, cc, row, col);
      const EpiIn<EPI>& x = in[p % RS][j];
      float v[VEC];
#pragma unroll
      for (int q = 0; q < VEC; ++q) v[q] = stg[r * EP + cc + q];
      if constexpr (sizeof(OutT) == 4) {
        if (split) {
          st_nt(W + (int64_t)row * g.N + col, make_float4(v[0], v[1], v[2], v[3]));
        } else {
          float* Cf = (float*)g.C + (int64_t)row * g.ldc + col;
          if (g.beta != 0.f) {
            const float4 old = *reinterpret_cast<const float4*>(Cf);
            v[0] += g.beta * old.x; v[1] += g.beta * old.y; v[2] += g.beta * old.z; v[3] += g.beta * old.w;
          }
          st_nt(Cf, make_float4(v[0], v[1], v[2], v[3]));
        }
      } else {
        bf16* Cb = (bf16*)g.C;
        const int64_t o = (int64_t)row * g.ldc + col;
        if constexpr (EPI == EPI_SWIGLU_BWD) {  // dz = v -> dgate | dup
          bf16x8 da, db;
#pragma unroll
          for (int q = 0; q < 8; ++q) {
            const float a = (float)x.a[q], bb = (float)x.b[q];
            const float sg = sigmoid_fast(a);
            da[q] = (bf16)(v[q] * bb * sg * (1.0f + a * (1.0f - sg)));
            db[q] = (bf16)(v[q] * a * sg);
          }
          st_nt(Cb + o, da);
          st_nt(Cb + o + g.N, db);
        } else if constexpr (EPI == EPI_DELTA) {  // dO, plus delta = rowsum(dO O) per head
          bf16x8 ov;
#pragma unroll
          for (int q = 0; q < 8; ++q) ov[q] = (bf16)v[q];
          st_nt(Cb + o, ov);
          float dot = 0.f;
#pragma unroll
          for (int q = 0; q < 8; ++q) dot += (float)ov[q] * (q < 4 ? x.o0[q] : x.o1[q - 4]);
          // the head's delta_hd / 8 chunks sit in consecutive lanes (aligned groups)
          for (int m = 1; m < g.delta_hd / 8; m <<= 1) dot += __shfl_xor(dot, m, 64);
          if (col % g.delta_hd == 0) {
            const int bb = row / g.delta_S, ii = row % g.delta_S, hh = col / g.delta_hd;
            g.delta[((int64_t)bb * (g.N / g.delta_hd) + hh) * g.delta_S + ii] = dot;
          }
        } else if constexpr (EPI == EPI_SWIGLU_FWD) {  // panel column col: gate or up of z column zc
          const int grp = col / 32, zc = (grp / 2) * 32 + col % 32;
          bf16x8 ov;
#pragma unroll
          for (int q = 0; q < 8; ++q) ov[q] = (bf16)v[q];
          bf16* Crow = Cb + (int64_t)row * g.ldc;
          if ((grp & 1) == 0) {
            st_nt(Crow + zc, ov);
            const float* up = stg + r * EP + cc + 32;  // the up values of the same z columns
            bf16x8 zv;
#pragma unroll
            for (int q = 0; q < 8; ++q) zv[q] = (bf16)(v[q] * sigmoid_fast(v[q]) * up[q]);
            st_nt((bf16*)g.out2 + (int64_t)row * g.ld_out2 + zc, zv);
          } else {
            st_nt(Crow + g.glu + zc, ov);
          }
        } else if constexpr (EPI == EPI_ROPE) {  // rotate pairs (i, i + hd/2) of each head
          bf16x8 ov;
          if (col < g.rope_cols) {
            const int hh = g.rope_hd / 2;
            const bool first = (col % g.rope_hd) < hh;
            const float* xp = stg + r * EP + (first ? cc + hh : cc - hh);  // partner columns
            const float cs[8] = {x.c0[0], x.c0[1], x.c0[2], x.c0[3], x.c1[0], x.c1[1], x.c1[2], x.c1[3]};
            const float sn[8] = {x.s0[0], x.s0[1], x.s0[2], x.s0[3], x.s1[0], x.s1[1], x.s1[2], x.s1[3]};
#pragma unroll
            for (int q = 0; q < 8; ++q)
              ov[q] = (bf16)(first ? v[q] * cs[q] - xp[q] * sn[q] : v[q] * cs[q] + xp[q] * sn[q]);
          } else {
#pragma unroll
            for (int q = 0; q < 8; ++q) ov[q] = (bf16)v[q];
          }
          st_nt(Cb + o, ov);
        } else if constexpr (EPI == EPI_AXPBY_DUP) {  // each value into two adjacent columns
          bf16x8 d0, d1;
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const bf16 u0 = (bf16)(g.alpha * v[q] + g.beta_d * (float)x.r[q]);
            const bf16 u1 = (bf16)(g.alpha * v[q + 4] + g.beta_d * (float)x.r[q + 4]);
            d0[2 * q] = u0; d0[2 * q + 1] = u0;
            d1[2 * q] = u1; d1[2 * q + 1] = u1;
          }
          bf16* Cd = Cb + (int64_t)row * g.ldc + 2 * col;
          st_nt(Cd, d0);
          st_nt(Cd + 8, d1);
        } else if constexpr (EPI == EPI_NS_SPLIT) {  // x = v + beta_d (hi + lo), then its hi/lo form
          bf16x8 h8, l8;
#pragma unroll
          for (int q = 0; q < 8; ++q) {
            const float xv = v[q] + g.beta_d * ((float)x.a[q] + (float)x.b[q]);
            const bf16 hq = (bf16)xv;
            h8[q] = hq;
            l8[q] = (bf16)(xv - (float)hq);
          }
          st_nt(Cb + o, h8);
          st_nt(Cb + o + g.N, l8);
        } else {
          if constexpr (EPI == EPI_RESID) {
#pragma unroll
            for (int q = 0; q < 8; ++q) v[q] += (float)x.r[q];
          } else if constexpr (EPI == EPI_AXPBY) {
#pragma unroll
            for (int q = 0; q < 8; ++q) v[q] = g.alpha * v[q] + g.beta_d * (float)x.r[q];
          }
          bf16x8 ov;
#pragma unroll
          for (int q = 0; q < 8; ++q) ov[q] = (bf16)v[q];
          st_nt(Cb + o, ov);
        }
      }
    }
    if constexpr (EPI == EPI_PLAIN && sizeof(OutT) == 2) {
      if (g.sym && m0 != n0) {
        // symmetric product, a tile above the diagonal: the part again at C[col, row], as 8-row
        // column segments of the staged rows
        constexpr int CT = WN * (RP / 8) / 64;  // segments per lane
        static_assert(CT * 64 == WN * (RP / 8), "every lane writes the same number of segments");
        bf16* Cb = (bf16*)g.C;
#pragma unroll
        for (int j = 0; j < CT; ++j) {
          const int c = lane + 64 * j, cc = c % WN, rg = c / WN;
          bf16x8 tv;
#pragma unroll
          for (int q = 0; q < 8; ++q) tv[q] = (bf16)stg[(rg * 8 + q) * EP + cc];
          const int row = m0 + wm0 + (p / NP) * 32 + RP * (p % NP) + rg * 8, col = n0 + wn0 + cc;
          st_nt(Cb + (int64_t)col * g.ldc + row, tv);
        }
      }
    }
    asm volatile("" ::: "memory");
  });
}

template <int BM, int BN, int WM, int WN, bool AK, bool BKM, typename OutT, bool CHECK>
__global__ void __launch_bounds__((BM / WM) * (BN / WN) * 64)
__attribute__((amdgpu_waves_per_eu(tile_waves_per_simd<BM, BN>(), tile_waves_per_simd<BM, BN>())))
gemm_mfma_kernel(GemmArgs g) {
  using C_ = Cfg<BM, BN, WM, WN, AK, BKM>;
  constexpr int WAVES_N = BN / WN;
  constexpr int NT = C_::NT, FM = C_::FM, FN = C_::FN, SA = C_::SA, SB = C_::SB;
  extern __shared__ __align__(16) unsigned char smem[];
  bf16* As = reinterpret_cast<bf16*>(smem);                 // [2][SA]
  bf16* Bs = As + 2 * SA;                                   // [2][SB]

  int m0, n0;
  tile_origin<BM, BN>(g, blockIdx.x, m0, n0);

  const int wave = threadIdx.x / 64, lane = threadIdx.x % 64;
  const int wm0 = (wave / WAVES_N) * WM, wn0 = (wave % WAVES_N) * WN;

  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  TileLoader<BM, NT, AK, CHECK> la;
  TileLoader<BN, NT, BKM, CHECK> lb;
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
  // Per k-slice, in this order (the compiler may not move instructions across the fences):
  //   step 0: global loads of the next slice, then the fragment reads of step 1, then the MFMAs
  //   steps 1, 2: fragment reads of the following step, then the MFMAs
  //   step 3: the MFMAs, each followed by its share of the LDS writes of the next slice
  // so every fragment read has a whole step of MFMAs to land, and the global loads three.
  constexpr int NM = FM * FN;
  constexpr int PA = decltype(la)::PER, PB = decltype(lb)::PER;
  constexpr int WPM = (PA + PB + NM - 1) / NM;  // LDS writes per MFMA in the last step
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    // next slice (the last iteration reloads its own slice, unused, so the loads and the LDS
    // writes are unconditional)
    const int kn = kbeg + min(kt + 1, nk - 1) * BK;
    const bf16* as = As + cur * SA;
    const bf16* bs = Bs + cur * SB;
    bf16* asn = As + (cur ^ 1) * SA;
    bf16* bsn = Bs + (cur ^ 1) * SB;
    bf16x8 af[2][FM], bfr[2][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i) af[0][i] = frag<BM, AK>(as, wm0 + i * 32, 0);
#pragma unroll
    for (int j = 0; j < FN; ++j) bfr[0][j] = frag<BN, BKM>(bs, wn0 + j * 32, 0);
    static_for<BK / 16>([&](auto KS) {
      constexpr int ks = KS, c = ks & 1;
      if constexpr (ks == 0) {
        la.load(A, g.lda, m0, g.M, kn, kend);
        lb.load(B, g.ldb, n0, g.N, kn, kend);
        __builtin_amdgcn_sched_barrier(0);
      }
      if constexpr (ks + 1 < BK / 16) {
#pragma unroll
        for (int i = 0; i < FM; ++i) af[c ^ 1][i] = frag<BM, AK>(as, wm0 + i * 32, (ks + 1) * 16);
#pragma unroll
        for (int j = 0; j < FN; ++j) bfr[c ^ 1][j] = frag<BN, BKM>(bs, wn0 + j * 32, (ks + 1) * 16);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
          for (int j = 0; j < FN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[c][i], bfr[c][j], acc[i][j], 0, 0, 0);
        __builtin_amdgcn_sched_barrier(0);
      } else {
        static_for<NM>([&](auto Q) {
          constexpr int q = Q, i = q / FN, j = q % FN;
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[c][i], bfr[c][j], acc[i][j], 0, 0, 0);
          static_for<WPM>([&](auto W) {
            constexpr int w = q * WPM + W;
            if constexpr (w < PA) la.store_one(asn, w);
            else if constexpr (w < PA + PB) lb.store_one(bsn, w - PA);
          });
          __builtin_amdgcn_sched_barrier(0);
        });
      }
    });
    __syncthreads();
  }

  gemm_epilogue<BM, BN, WM, WN, OutT, CHECK>(g, acc, reinterpret_cast<float*>(smem), m0, n0, wm0, wn0);
}

// ---------------------------------------------------------------------------------------------
// Full-tile kernel with direct-to-LDS operand loads (gfx950 global_load_lds_dwordx4): each lane's
// 16 bytes land at the wave's LDS base + 16 * lane, so a tile is written in lane order and the
// bank spreading is an XOR swizzle of 16-byte chunks instead of padding:
//   k-contiguous tile [ROWS][BKT]: chunk kc of row r sits at r * BKT/8 + (kc ^ ((r / (128/BKT)) mod
//     BKT/8)), so the 16 rows one 16-lane group reads for a fragment cover all 64 banks;
//   row-contiguous tile [BKT][ROWS]: chunk rc of k-row k sits at k * ROWS/8 + (rc ^ 4 (k mod 4)), so
//     the 4 k-rows x 32 rows of one half-wave transposing read fall in 4 different 64-byte bank
//     groups (ROWS >= 128, a whole number of 256-byte bank periods per k-row).
// NS stages: the loads of slice kt + NS - 1 are issued while slice kt is consumed, so a load has
// NS - 1 slices of MFMAs to land; one barrier per slice, after each thread has seen its own loads
// of the slice complete (vmcnt), makes every thread's loads of it visible.
template <int ROWS, int BKT, bool KMAJ, int NT>
struct DmaTile {
  static constexpr int CHUNKS = ROWS * BKT / 8;
  static constexpr int PER = CHUNKS / NT;  // loads per thread and slice
  static constexpr int ELEMS = ROWS * BKT;
  static_assert(CHUNKS % NT == 0, "tile does not split evenly over the threads");
  static_assert(KMAJ || ROWS >= 128, "row-contiguous swizzle needs 256-byte k-rows");
  // k-contiguous tile: the row and the 8-element k chunk whose data LDS chunk p holds
  __device__ static void row_chunk(int p, int& r, int& kc) {
    constexpr int CPR = BKT / 8, RPB = 128 / BKT;
    r = p / CPR;
    kc = (p % CPR) ^ ((r / RPB) % CPR);
  }
  // element offset, from the tile origin in global memory, of the data for LDS chunk p
  __device__ static int64_t src(int p, int ld) {
    if constexpr (KMAJ) {
      constexpr int CPR = BKT / 8, RPB = 128 / BKT;
      const int r = p / CPR, kc = (p % CPR) ^ ((r / RPB) % CPR);
      return (int64_t)r * ld + kc * 8;
    } else {
      constexpr int CPK = ROWS / 8;
      const int k = p / CPK, rc = (p % CPK) ^ (4 * (k & 3));
      return (int64_t)k * ld + rc * 8;
    }
  }
  // MFMA fragment: row r0 + lane mod 32, k = k0 + 8 (lane / 32) .. +7
  __device__ static bf16x8 frag(const bf16* T, int r0, int k0) {
    const int l = threadIdx.x % 64;
    if constexpr (KMAJ) {
      constexpr int CPR = BKT / 8, RPB = 128 / BKT;
      const int r = r0 + l % 32, kc = k0 / 8 + l / 32;
      return *reinterpret_cast<const bf16x8*>(T + r * BKT + ((kc ^ ((r / RPB) % CPR)) << 3));
    } else {
      const int gq = l / 16, i = l % 16;
      const int r = r0 + 16 * (gq & 1) + 4 * (i & 3);
      const int k = k0 + 8 * (gq >> 1) + (i >> 2);  // k and k + 4 share k mod 4
      const int col = (((r >> 3) ^ (4 * (k & 3))) << 3) + (r & 7);
      typedef __attribute__((address_space(3))) v4i16_t lds_v4i16;
      const v4i16_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(T + k * ROWS + col));
      const v4i16_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(T + (k + 4) * ROWS + col));
      bf16x8 f;
      __builtin_memcpy(&f, &lo, 8);
      __builtin_memcpy(reinterpret_cast<char*>(&f) + 8, &hi, 8);
      return f;
    }
  }
};

template <int BM, int BN, int WM, int WN, bool AK, bool BKM, int BKT, int NS>
struct DmaCfg {
  static constexpr int NW = (BM / WM) * (BN / WN);
  static constexpr int NT = NW * 64;
  using TA = DmaTile<BM, BKT, AK, NT>;
  using TB = DmaTile<BN, BKT, BKM, NT>;
  // one stage: the A tile, then the B tile (bf16 elements)
  static constexpr int STAGE = TA::ELEMS + TB::ELEMS;
  // epilogue staging rows per part: 16 when that fits in one stage, else 8
  static constexpr int RP = (size_t)NW * 16 * (WN + 4) * sizeof(float) <= (size_t)STAGE * sizeof(bf16) ? 16 : 8;
  static constexpr size_t epi_lds = (size_t)NW * RP * (WN + 4) * sizeof(float);
  // A block walks several tiles when the epilogue's staging fits in one stage: the stage of a
  // tile's last slice is then free for it while the next tile's first slices land in the others.
  static constexpr bool persist = epi_lds <= (size_t)STAGE * sizeof(bf16);
  static constexpr size_t main_lds = (size_t)NS * STAGE * sizeof(bf16);
  static constexpr size_t lds = main_lds > epi_lds ? main_lds : epi_lds;
};

// waves per SIMD: the block's waves over the 4 SIMDs times the blocks the LDS lets a CU hold
template <int BM, int BN, int WM, int WN, bool AK, bool BKM, int BKT, int NS>
constexpr int dma_waves_per_simd() {
  using C_ = DmaCfg<BM, BN, WM, WN, AK, BKM, BKT, NS>;
  const int blocks = (int)(163840 / C_::lds);
  const int w = (C_::NW / 4) * (blocks > 0 ? blocks : 1);
  return w > 8 ? 8 : (w < 1 ? 1 : w);
}

// Block b takes tiles b, b + gridDim.x, ... (gridDim.x a multiple of 8 when it is below the tile
// count, so that every tile of a block maps to the block's XCD).  The slices of all its tiles form
// one sequence: the loads of slice G + NS - 1 of that sequence (the next tile's first slices near
// the end of a tile) are issued while slice G is consumed, into stage (G + NS - 1) mod NS.
template <int BM, int BN, int WM, int WN, bool AK, bool BKM, typename OutT, int BKT, int NS, int EPI>
__global__ void __launch_bounds__((BM / WM) * (BN / WN) * 64)
__attribute__((amdgpu_waves_per_eu(dma_waves_per_simd<BM, BN, WM, WN, AK, BKM, BKT, NS>(),
                                   dma_waves_per_simd<BM, BN, WM, WN, AK, BKM, BKT, NS>())))
gemm_dma_kernel(GemmArgs g) {
  if (g.batch > 1) {  // product blockIdx.z of a batch
    const int64_t z = blockIdx.z;
    g.A = (const bf16*)g.A + z * g.sA;
    g.B = (const bf16*)g.B + z * g.sB;
    g.C = (char*)g.C + z * g.sC * (int64_t)sizeof(OutT);
    if (g.D) g.D = (const OutT*)g.D + z * g.sD;
  }
  using C_ = DmaCfg<BM, BN, WM, WN, AK, BKM, BKT, NS>;
  using TA = typename C_::TA;
  using TB = typename C_::TB;
  constexpr int WAVES_N = BN / WN, NW = C_::NW, STAGE = C_::STAGE;
  constexpr int FM = WM / 32, FN = WN / 32;
  constexpr int PA = TA::PER, PB = TB::PER;
  // vector-memory operations one thread's epilogue issues at least: one per 16-byte output chunk
  constexpr int RP = C_::RP, CPP = RP * WN / (sizeof(OutT) == 2 ? 8 : 4);  // 16-byte chunks per part
  static_assert(CPP % 64 == 0, "every lane stores the same number of chunks per part");
  constexpr int EPI_OPS = FM * (32 / RP) * (CPP / 64);
  static_assert((NS - 2) * (PA + PB) + EPI_OPS < 64, "vmcnt range");
  extern __shared__ __align__(16) unsigned char smem[];
  bf16* S = reinterpret_cast<bf16*>(smem);  // [NS][A tile | B tile]

  const int tiles = g.sym ? (g.M / BM) * (g.M / BM + 1) / 2 : (g.M / BM) * (g.N / BN);
  auto origin = [&](int b, int& m0_, int& n0_) {
    if (g.sym) tri_origin<BM, BN>(g, b, m0_, n0_);
    else tile_origin<BM, BN>(g, b, m0_, n0_);
  };
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / 64), lane = threadIdx.x % 64;
  const int wm0 = (wave / WAVES_N) * WM, wn0 = (wave % WAVES_N) * WN;
  // split-K: this block covers slices [s0, s0 + nk) of every tile
  const int nk = g.K / BKT / g.ksplit, s0 = blockIdx.y * nk;
  const bool glu = BKM && EPI == EPI_SWIGLU_FWD;
  // this thread's byte offsets from a tile's slice origin
  uint32_t oa[PA], ob[PB];
#pragma unroll
  for (int q = 0; q < PA; ++q) oa[q] = 2u * (uint32_t)TA::src((q * NW + wave) * 64 + lane, g.lda);
#pragma unroll
  for (int q = 0; q < PB; ++q) {
    const int p = (q * NW + wave) * 64 + lane;
    if (glu) {
      // epilogue 3: panel row n0 + r is gate row (or, in odd 32-row groups, up row) n0/2 + ...
      int r, kc;
      TB::row_chunk(p, r, kc);
      ob[q] = 2u * (uint32_t)((((r / 32) & 1) * g.glu + (r / 64) * 32 + r % 32) * g.ldb + kc * 8);
    } else {
      ob[q] = 2u * (uint32_t)TB::src(p, g.ldb);
    }
  }
  // slice 0 (of this split) of the tiles at row m0 / column n0
  auto a_tile = [&](int m0) {
    return (const bf16*)g.A + (AK ? (int64_t)m0 * g.lda + (int64_t)s0 * BKT : (int64_t)s0 * BKT * g.lda + m0);
  };
  auto b_tile = [&](int n0) {
    if (glu) return (const bf16*)g.B + (int64_t)(n0 / 2) * g.ldb + (int64_t)s0 * BKT;
    return (const bf16*)g.B + (BKM ? (int64_t)n0 * g.ldb + (int64_t)s0 * BKT : (int64_t)s0 * BKT * g.ldb + n0);
  };
  const int64_t step_a = AK ? BKT : (int64_t)BKT * g.lda;
  const int64_t step_b = BKM ? BKT : (int64_t)BKT * g.ldb;
  // LDS byte addresses of this wave's first chunk of the A and B tiles of stage 0
  typedef __attribute__((address_space(3))) bf16 lds_bf16;
  const uint32_t la0 = (uint32_t)(uintptr_t)(lds_bf16*)(S + wave * 512);
  const uint32_t lb0 = la0 + TA::ELEMS * 2;
  auto issue = [&](const bf16* at, const bf16* bt, int s, int stage) {
    const bf16* as = at + s * step_a;
    const bf16* bs = bt + s * step_b;
    const uint32_t ta = la0 + stage * STAGE * 2, tb = lb0 + stage * STAGE * 2;
#pragma unroll
    for (int q = 0; q < PA; ++q) dma16(as, oa[q], ta + q * NW * 1024);
#pragma unroll
    for (int q = 0; q < PB; ++q) dma16(bs, ob[q], tb + q * NW * 1024);
  };

  int t = blockIdx.x;
  int m0, n0;
  origin(t, m0, n0);
  const bf16* at = a_tile(m0);
  const bf16* bt = b_tile(n0);
  // slices NS - 1 and later ahead come from the next tile only when a tile has that many
  const bool chain = C_::persist && nk >= NS - 1;
#pragma unroll
  for (int s = 0; s < NS - 1; ++s) issue(at, bt, min(s, nk - 1), s);
  int G = 0;  // position in the block's slice sequence
  for (bool first = true;; first = false) {
    const int tn = t + gridDim.x;
    const bool next = chain && tn < tiles;
    int m1 = m0, n1 = n0;
    if (next) origin(tn, m1, n1);
    const bf16* atn = a_tile(m1);
    const bf16* btn = b_tile(n1);

    f32x16 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

    for (int kt = 0; kt < nk; ++kt, ++G) {
      // this thread's loads of slice G are in LDS: issued after them are the loads of the NS - 2
      // following slices and, in a tile's first slices, the previous tile's epilogue
      if (!first && kt < NS - 1) wait_vm_lds<(NS - 2) * (PA + PB) + EPI_OPS>();
      else wait_vm_lds<(NS - 2) * (PA + PB)>();
      block_barrier();  // ... and every thread's; the stage of slice G - 1 is free
      {
        const int x = kt + NS - 1, stage = (G + NS - 1) % NS;
        if (x < nk) issue(at, bt, x, stage);
        else if (next) issue(atn, btn, x - nk, stage);
        else issue(at, bt, nk - 1, stage);  // a reload into a stage nobody reads again
      }
      const bf16* as = S + (G % NS) * STAGE;
      const bf16* bs = as + TA::ELEMS;
      bf16x8 af[2][FM], bfr[2][FN];
#pragma unroll
      for (int i = 0; i < FM; ++i) af[0][i] = TA::frag(as, wm0 + i * 32, 0);
#pragma unroll
      for (int j = 0; j < FN; ++j) bfr[0][j] = TB::frag(bs, wn0 + j * 32, 0);
      // the next k-step's fragment reads go out between this step's MFMAs (one read after each
      // MFMA; they write the other fragment buffer), so the LDS and matrix pipes work together
      static_for<BKT / 16>([&](auto KS) {
        constexpr int ks = KS, c = ks & 1;
        __builtin_amdgcn_sched_barrier(0);
        if constexpr (ks + 1 < BKT / 16) {
#pragma unroll
          for (int i = 0; i < FM; ++i) af[c ^ 1][i] = TA::frag(as, wm0 + i * 32, (ks + 1) * 16);
#pragma unroll
          for (int j = 0; j < FN; ++j) bfr[c ^ 1][j] = TB::frag(bs, wn0 + j * 32, (ks + 1) * 16);
        }
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
          for (int j = 0; j < FN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[c][i], bfr[c][j], acc[i][j], 0, 0, 0);
        if constexpr (ks + 1 < BKT / 16) {
          static_assert(FM * FN >= FM + FN, "one MFMA ahead of every fragment read");
          static_for<FM + FN>([&](auto) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // one LDS read
          });
          __builtin_amdgcn_sched_group_barrier(0x008, FM * FN - (FM + FN), 0);
        }
        __builtin_amdgcn_sched_barrier(0);
      });
    }
    float* stg;
    if constexpr (C_::persist) {
      // the stage of the tile's last slice, once every wave is past its fragment reads
      stg = reinterpret_cast<float*>(S + ((G - 1) % NS) * STAGE);
    } else {
      wait_vm_lds<0>();  // the whole LDS: the reloads too
      stg = reinterpret_cast<float*>(smem);
    }
    wait_vm_lds<63>();
    block_barrier();
    dma_epilogue<BM, BN, WM, WN, OutT, EPI, C_::RP>(g, acc, stg, m0, n0, wm0, wn0);
    if (!next) break;
    t = tn; m0 = m1; n0 = n1; at = atn; bt = btn;
  }
  wait_vm_lds<0>();  // no load may land in the LDS after the block ends
}

// C = beta C + sum over splits of the partial tiles, in split order (fp32 output, ldc == N)
__global__ void __launch_bounds__(256) splitk_reduce(const float* __restrict__ ws, int splits, int64_t mn,
                                                     float* __restrict__ C, float beta) {
  const int64_t i = 4 * ((int64_t)blockIdx.x * blockDim.x + threadIdx.x);
  if (i >= mn) return;
  if (i + 3 < mn) {
    float4 acc = ld_nt<float4>(ws + i);
    for (int s = 1; s < splits; ++s) {
      const float4 v = ld_nt<float4>(ws + (int64_t)s * mn + i);
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

template <int BM, int BN, int WM, int WN, bool AK, bool BKM, typename OutT, bool CHECK>
void launch_one(const GemmArgs& g, int nblk, hipStream_t st) {
  using C_ = Cfg<BM, BN, WM, WN, AK, BKM>;
  static bool attr_set = false;
  if (!attr_set) {
    (void)hipFuncSetAttribute((const void*)gemm_mfma_kernel<BM, BN, WM, WN, AK, BKM, OutT, CHECK>,
                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)C_::lds);
    attr_set = true;
  }
  gemm_mfma_kernel<BM, BN, WM, WN, AK, BKM, OutT, CHECK><<<dim3(nblk, g.ksplit), C_::NT, C_::lds, st>>>(g);
}

template <int BM, int BN, int WM, int WN, typename OutT>
void launch_cfg(const GemmArgs& g, hipStream_t st) {
  const int nblk = (int)(cdiv(g.M, BM) * cdiv(g.N, BN));
  // full tiles and whole k-slices everywhere (each split covers a whole number of slices)
  const bool even = g.M % BM == 0 && g.N % BN == 0 && g.K % BK == 0 &&
                    (g.ksplit == 1 || (g.K / BK) % g.ksplit == 0);
#define L(AK, BKM)                                                                        \
  do {                                                                                    \
    if (even) launch_one<BM, BN, WM, WN, AK, BKM, OutT, false>(g, nblk, st);              \
    else launch_one<BM, BN, WM, WN, AK, BKM, OutT, true>(g, nblk, st);                    \
  } while (0)
  if (g.a_kmajor && g.b_kmajor) L(true, true);
  else if (g.a_kmajor) L(true, false);
  else if (g.b_kmajor) L(false, true);
  else L(false, false);
#undef L
}

template <int BM, int BN, int WM, int WN, bool AK, bool BKM, typename OutT, int BKT, int NS, int EPI>
void launch_dma_one(const GemmArgs& g, int nblk, hipStream_t st) {
  using C_ = DmaCfg<BM, BN, WM, WN, AK, BKM, BKT, NS>;
  static bool attr_set = false;
  if (!attr_set) {
    (void)hipFuncSetAttribute((const void*)gemm_dma_kernel<BM, BN, WM, WN, AK, BKM, OutT, BKT, NS, EPI>,
                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)C_::lds);
    attr_set = true;
  }
  // more tiles than the chip holds blocks at once: one block per slot, each walking its tiles
  int grid = nblk;
  if (C_::persist && g.batch == 1 && g.K / BKT / g.ksplit >= NS - 1) {
    const int per_cu = (int)(163840 / C_::lds);
    const int slots = (per_cu * device_cu_count() / g.ksplit) / 8 * 8;
    if (slots >= 8 && nblk > slots) grid = slots;
  }
  gemm_dma_kernel<BM, BN, WM, WN, AK, BKM, OutT, BKT, NS, EPI><<<dim3(grid, g.ksplit, g.batch), C_::NT, C_::lds, st>>>(g);
}

// Direct-to-LDS variant: full tiles and whole slices per split only; false if the shape is not.
// fp32 output: every operand layout, no fused epilogue; bf16 output: a k-contiguous A (every
// bf16-output product of the stage has one) with each epilogue kind.
template <int BM, int BN, int WM, int WN, typename OutT, int BKT, int NS>
bool launch_dma_cfg(const GemmArgs& g, hipStream_t st) {
  if (g.M % BM || g.N % BN || g.K % BKT || g.K == 0 || (g.K / BKT) % g.ksplit) return false;
  if (g.sym && (BM != BN || g.M != g.N || g.epi != 0 || g.resid || sizeof(OutT) != 2)) return false;
  const int nblk = g.sym ? (g.M / BM) * (g.M / BM + 1) / 2 : (g.M / BM) * (g.N / BN);
  if constexpr (sizeof(OutT) == 4) {
    if (g.a_kmajor && g.b_kmajor) launch_dma_one<BM, BN, WM, WN, true, true, OutT, BKT, NS, EPI_PLAIN>(g, nblk, st);
    else if (g.a_kmajor) launch_dma_one<BM, BN, WM, WN, true, false, OutT, BKT, NS, EPI_PLAIN>(g, nblk, st);
    else if (g.b_kmajor) launch_dma_one<BM, BN, WM, WN, false, true, OutT, BKT, NS, EPI_PLAIN>(g, nblk, st);
    else launch_dma_one<BM, BN, WM, WN, false, false, OutT, BKT, NS, EPI_PLAIN>(g, nblk, st);
  } else {
    if (!g.a_kmajor) return false;
    const int kind = g.epi != 0 ? g.epi : (g.resid ? EPI_RESID : EPI_PLAIN);
#define K_(E)                                                                                     \
  case E:                                                                                         \
    if (g.b_kmajor) launch_dma_one<BM, BN, WM, WN, true, true, OutT, BKT, NS, E>(g, nblk, st);     \
    else launch_dma_one<BM, BN, WM, WN, true, false, OutT, BKT, NS, E>(g, nblk, st);              \
    break;
    switch (kind) {
      K_(EPI_PLAIN) K_(EPI_SWIGLU_BWD) K_(EPI_ROPE) K_(EPI_SWIGLU_FWD) K_(EPI_DELTA) K_(EPI_RESID)
      K_(EPI_AXPBY) K_(EPI_AXPBY_DUP) K_(EPI_NS_SPLIT)
      default: return false;
    }
#undef K_
  }
  return true;
}

}  // namespace

namespace {
// Tile choice for full tiles: 256 x 256 (8 waves of 64 x 128, 64-deep slices in 2 stages) when the
// product has enough of them and is deep enough for the larger tile to pay (at K = 768 the
// persistent 128 x 128 kernel is faster, from K = 1536 on the 256 x 256 one), else 128 x 128.
constexpr int BIG_K = 1536;
bool use_big(const GemmArgs& g) {
  const int64_t t256 = cdiv(g.M, 256) * cdiv(g.N, 256);
  return g.M % 256 == 0 && g.N % 256 == 0 && g.K % 64 == 0 && g.K >= BIG_K &&
         (t256 >= 512 || (t256 >= 256 && g.K >= 2048));
}
}  // namespace

int device_cu_count() {
  static int cus[64] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (cus[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    cus[dev] = n;
  }
  return cus[dev];
}

bool gemm_mfma_try(const GemmArgs& g0, hipStream_t st) {
  // vector-load alignment: 8 elements along every contiguous dimension, rows in groups of 4
  if (g0.K % 8 || g0.M % 8 || g0.N % 8 || g0.lda % 8 || g0.ldb % 8 || g0.ldc % 8) return false;
  if (g0.batch > 1 || g0.sym || g0.epi == EPI_AXPBY || g0.epi == EPI_AXPBY_DUP || g0.epi == EPI_NS_SPLIT) {
    // batched and AXPBY products run on the direct-to-LDS kernels only (full tiles, 16-byte
    // aligned operands and batch strides; AXPBY with bf16 output, fp32 output plain or
    // accumulating beta C); the caller loops over the others
    const bool ok = g0.a_kmajor && g0.M % 128 == 0 && g0.N % 128 == 0 && g0.K % 64 == 0 &&
                    (g0.epi == 0 || ((g0.epi == EPI_AXPBY || g0.epi == EPI_AXPBY_DUP || g0.epi == EPI_NS_SPLIT) &&
                                     !g0.out_f32)) && !g0.resid &&
                    ((uintptr_t)g0.A | (uintptr_t)g0.B | (uintptr_t)g0.C | (uintptr_t)g0.D) % 16 == 0 &&
                    (g0.sA | g0.sB | g0.sC | g0.sD) % 8 == 0 &&
                    (!g0.sym || (g0.M == g0.N && g0.epi == 0 && !g0.out_f32));
    if (!ok) return false;
    GemmArgs g = g0;
    g.ksplit = 1;
    return g.out_f32 ? launch_dma_cfg<128, 128, 64, 64, float, 64, 2>(g, st)
                     : launch_dma_cfg<128, 128, 64, 64, bf16, 64, 2>(g, st);
  }
  if (g0.epi == 3) {
    // the SwiGLU forward rides in the epilogue of the direct-to-LDS kernels only (their B loader
    // gathers gate and up rows); any other shape runs the product, then the SwiGLU kernel
    const bool fused = !g0.out_f32 && g0.b_kmajor && g0.K > 0 && g0.K % 64 == 0 && g0.M % 128 == 0 &&
                       g0.N == 2 * g0.glu && g0.glu % 64 == 0 && g0.ld_out2 % 8 == 0 &&
                       (uintptr_t)g0.out2 % 16 == 0;
    if (!fused) {
      GemmArgs p = g0;
      p.epi = 0;
      p.glu = 0;
      if (!gemm_mfma_try(p, st)) return false;
      launch_swiglu_fwd(true, g0.C, g0.out2, g0.M, g0.glu, st);
      return true;
    }
  }
  if (g0.epi == 1 && (g0.out_f32 || g0.ld_aux % 8 || (uintptr_t)g0.aux % 16)) return false;
  if ((uintptr_t)g0.A % 16 || (uintptr_t)g0.B % 16 || (uintptr_t)g0.C % 16 || (uintptr_t)g0.resid % 16)
    return false;
  if (g0.epi == 4) {
    // delta rides in the epilogue of the direct-to-LDS kernels when a wave's columns hold whole
    // heads (every lane of the epilogue active); otherwise the caller computes it separately
    const bool full = !g0.out_f32 && g0.K > 0 && g0.K % 64 == 0 && g0.M % 128 == 0 && g0.N % 128 == 0;
    const int wn = full && use_big(g0) ? 128 : 64;
    if (!full || g0.delta_hd < 8 || wn % g0.delta_hd || g0.ld_aux % 8 || (uintptr_t)g0.aux % 16) return false;
  }
  GemmArgs g = g0;
  g.ksplit = 1;
  const int64_t mn = (int64_t)g.M * g.N;
  // Full tiles go to the direct-to-LDS kernels (use_big picks 256 x 256 or 128 x 128: 4 waves,
  // 64-deep slices in 2 stages, two blocks per CU, persistent when the tiles outnumber the
  // blocks the chip holds); ragged shapes to the register-staged kernel with bounds-checked loads.
  constexpr int DKB = 64, DKS = 64;
  const bool full128 = g.M % 128 == 0 && g.N % 128 == 0 && g.K % DKS == 0;
  const int64_t t256 = cdiv(g.M, 256) * cdiv(g.N, 256), t128 = cdiv(g.M, 128) * cdiv(g.N, 128);
  const bool big = use_big(g);
  const int64_t tiles = big ? t256 : t128;
  if (g.out_f32 && g.ws && g.ldc == g.N && tiles < 512 && g.K >= 2048) {
    // deterministic split-K for underfilled fp32-output products: whole slices per split
    const int kq = big ? DKB : (full128 ? DKS : BK);
    int s = (int)std::min<int64_t>(8, cdiv(512, tiles));
    while (s > 1 && (s * mn > g.ws_elems || g.K / s < 512 || (g.K / kq) % s)) --s;
    g.ksplit = s;
  }
  // RoPE in the epilogue needs every head whole inside one wave's columns
  const int wn = big ? 128 : 64;
  const bool rope_after = g.epi == 2 && (g.out_f32 || wn % g.rope_hd != 0);
  if (rope_after) g.epi = 0;
  bool done = false;  // the direct-to-LDS launchers decline shapes they do not take (K = 0)
  if (big)
    done = g.out_f32 ? launch_dma_cfg<256, 256, 64, 128, float, DKB, 2>(g, st)
                     : launch_dma_cfg<256, 256, 64, 128, bf16, DKB, 2>(g, st);
  else if (full128)
    done = g.out_f32 ? launch_dma_cfg<128, 128, 64, 64, float, DKS, 2>(g, st)
                     : launch_dma_cfg<128, 128, 64, 64, bf16, DKS, 2>(g, st);
  if (!done) {
    if (g.out_f32) launch_cfg<128, 128, 64, 64, float>(g, st);
    else launch_cfg<128, 128, 64, 64, bf16>(g, st);
  }
  if (g.ksplit > 1)
    splitk_reduce<<<(unsigned)cdiv(cdiv(mn, 4), 256), 256, 0, st>>>(g.ws, g.ksplit, mn, (float*)g.C, g.beta);
  if (rope_after)
    launch_rope(!g.out_f32, g.C, g.M, g.rope_S, g.rope_cols / g.rope_hd, g.rope_hd, g.ldc, g.rope_cos,
                g.rope_sin, false, st);
  return true;
}
