// Causal grouped-query flash attention on gfx950 matrix cores (bf16 in, fp32 accumulation).
//
// Every LDS tile holds rows of a head as they sit in memory ([row][d], 16-byte copies), unpadded,
// with the 16-byte chunks of row r permuted by an XOR with swz(r) so that both ways of reading a
// tile are free of bank conflicts (64 banks; a 16-byte read is served 16 lanes, an 8-byte read half
// a wave, per cycle).  The MFMA operand v_mfma_f32_32x32x16_bf16 wants 8 consecutive contraction
// values per lane:
//   - contraction over d (S = Q K^T, dP = dO V^T): 16-byte reads of a row;
//   - contraction over rows (O^T += V^T P^T, dQ^T += K^T dS^T, dV^T += dO^T P, dK^T += Q^T dS):
//     two ds_read_b64_tr_b16 transposing reads (each 16-lane group reads a 4 x 16 block whose
//     column j lands in lane j).
// Forward, per (batch, query head, block of 128 queries), each of the 4 waves owning 32 queries:
//   S^T = K Q^T (B = the wave's Q rows in registers) -> lane l owns query column l mod 32, so the
//   online-softmax statistics of a query stay in one lane pair (l, l ^ 32); O^T += V^T P^T with P^T
//   rebuilt from the S^T accumulators by one lane-pair exchange; lse = ln sum exp(S) is kept.
// Backward (dS = P (dP - delta), delta = rowsum(dO O) with O in fp32, P recomputed from lse), two
// kernels and no float atomics: dQ (waves own queries, K and V tiles streamed) and dK/dV (waves own keys, Q and
// dO tiles of every query head of the key/value head streamed).  Tiles are double-buffered through
// registers: the next tile is fetched while the current one feeds the MFMAs.  Outputs leave through
// LDS as 16-byte rows.  Query blocks with the longest causal range are scheduled first.
#include "common.h"
#include "kernels.h"
#include <algorithm>

namespace {

constexpr int QB = 128;   // queries (forward, dQ) or keys (dK/dV) per workgroup
constexpr int KB = 64;    // rows per streamed tile
constexpr int NT = 256;   // 4 waves
constexpr float LOG2E = 1.4426950408889634f;


typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
// two floats -> two RNE bf16 in one dword (a in the low half): one v_cvt_pk_bf16_f32
__device__ __forceinline__ uint32_t pack2(float a, float b) {
  const bf16x2 v = __builtin_convertvector((f32x2){a, b}, bf16x2);
  uint32_t u;
  __builtin_memcpy(&u, &v, 4);
  return u;
}

// Chunk permutation of tile row r (HD/8 chunks of 16 bytes per row):
//   HD = 128 (a row spans the 64 banks): swz = 4 (r mod 4) + (r / 4 mod 4), a bijection on any 16
//     consecutive rows (16-byte row reads) that sends 4 consecutive rows (k0 a multiple of 4) to 4
//     different 4-chunk groups (transposing reads of 4 rows x 32 columns);
//   HD = 64 (two rows per 64 banks): swz = 4 (r / 2 mod 2) + (r / 4 mod 4), the same two properties
//     over the rows of one parity.
template <int HD>
__device__ __forceinline__ int swz(int r) {
  if constexpr (HD == 128) return 4 * (r & 3) + ((r >> 2) & 3);
  else return 4 * ((r >> 1) & 1) + ((r >> 2) & 3);
}
// element index of (row r, column c) in a swizzled [row][HD] tile
template <int HD>
__device__ __forceinline__ int tidx(int r, int c) {
  return r * HD + ((((c >> 3) ^ swz<HD>(r))) << 3) + (c & 7);
}

// fragment of a [row][k] tile: row r0 + lane mod 32, k = k0 + 8 (lane / 32) .. +7
template <int HD>
__device__ __forceinline__ bf16x8 frag_rows(const bf16* T, int r0, int k0) {
  const int l = threadIdx.x % 64;
  return *reinterpret_cast<const bf16x8*>(T + tidx<HD>(r0 + l % 32, k0 + 8 * (l / 32)));
}

// fragment of the transpose of a [k][col] tile: col c0 + lane mod 32, k = k0 + 8 (lane / 32) .. +7,
// from two transposing reads (each 16-lane group reads 4 rows x 16 columns; lane j gets column j)
template <int HD>
__device__ __forceinline__ bf16x8 frag_cols(const bf16* T, int c0, int k0) {
  const int l = threadIdx.x % 64, g = l / 16, i = l % 16;
  const int c = c0 + 16 * (g & 1) + 4 * (i & 3);
  const int k = k0 + 8 * (g >> 1) + (i >> 2);
  typedef __attribute__((address_space(3))) v4i16_t lds_v4i16;
  const v4i16_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(T + tidx<HD>(k, c)));
  const v4i16_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(T + tidx<HD>(k + 4, c)));
  bf16x8 f;
  __builtin_memcpy(&f, &lo, 8);
  __builtin_memcpy(reinterpret_cast<char*>(&f) + 8, &hi, 8);
  return f;
}

// gfx950 v_permlane32_swap(X, Y) exchanges lanes 32..63 of X with lanes 0..31 of Y (no LDS trip).
__device__ __forceinline__ void swap32(uint32_t& x, uint32_t& y) {
  const auto r = __builtin_amdgcn_permlane32_swap(x, y, false, false);
  x = r[0];
  y = r[1];
}
// v combined with the value of lane l ^ 32: after swap32(a, a) the two results are v and the
// partner's value in some order, so a commutative op of the two gives the same value on both lanes
__device__ __forceinline__ float pair_max(float v) {
  uint32_t a = __float_as_uint(v), b = a;
  swap32(a, b);
  return fmaxf(__uint_as_float(a), __uint_as_float(b));
}
__device__ __forceinline__ float pair_sum(float v) {
  uint32_t a = __float_as_uint(v), b = a;
  swap32(a, b);
  return __uint_as_float(a) + __uint_as_float(b);
}

// B operand (8 consecutive k at column lane mod 32) from a 32x32 accumulator whose rows are the k
// index, for the 16-row group starting at accumulator index ib (0 or 8).  Lane half h holds rows
// ib+4h..ib+4h+3 of the group; the operand wants rows 8h..8h+7: half 0 needs its own rows ib..ib+3
// then its partner's, half 1 its partner's rows ib+4..ib+7 then its own.  Swapping the packed lower
// pair (lanes 32..63) with the packed upper pair (lanes 0..31) leaves exactly that in every lane:
// the first word of each swap is the operand's first half, the second word its second half.
template <int IB>
__device__ __forceinline__ bf16x8 acc_rows_to_b(const f32x16& s) {
  uint32_t lo0 = pack2(s[IB + 0], s[IB + 1]), lo1 = pack2(s[IB + 2], s[IB + 3]);
  uint32_t hi0 = pack2(s[IB + 4], s[IB + 5]), hi1 = pack2(s[IB + 6], s[IB + 7]);
  swap32(lo0, hi0);
  swap32(lo1, hi1);
  const uint32_t pw[4] = {lo0, lo1, hi0, hi1};
  bf16x8 r;
  __builtin_memcpy(&r, pw, 16);
  return r;
}

// The same operand from an accumulator split in two: hi = bf16(s) and lo = bf16(s - hi), so that
// a product with hi and one with lo add up to the product with s to about 2^-17 relative (s - hi is
// exact in fp32).
template <int IB>
__device__ __forceinline__ void acc_rows_to_b_split(const f32x16& s, bf16x8& hi, bf16x8& lo) {
  uint32_t h[4], l[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const float a = s[IB + 2 * q], b = s[IB + 2 * q + 1];
    h[q] = pack2(a, b);
    l[q] = pack2(a - __uint_as_float(h[q] << 16), b - __uint_as_float(h[q] & 0xffff0000u));
  }
  swap32(h[0], h[2]);
  swap32(h[1], h[3]);
  swap32(l[0], l[2]);
  swap32(l[1], l[3]);
  __builtin_memcpy(&hi, h, 16);
  __builtin_memcpy(&lo, l, 16);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Streamed tiles: KB rows x HD of a head (row stride ld) land in a swizzled [KB][HD] LDS tile by
// direct-to-LDS loads.  Load q of a wave writes 1 KB (16 bytes per lane, in lane order), so LDS
// chunk p = (q * 4 + wave) * 64 + lane of the tile holds row p / (HD/8), data chunk
// (p mod HD/8) ^ swz(row): the layout tidx reads.  Rows at or beyond the tile's valid rows repeat
// its last valid row (finite data whose probabilities the causal mask makes exactly zero).
template <int HD>
struct DmaRowTile {
  static constexpr int CPR = HD / 8;
  static constexpr int PER = KB * CPR / NT;  // loads per thread and tile
  static_assert(PER * NT == KB * CPR, "tile does not split evenly over the threads");
  // byte offset, from the tile's first row in global memory, of this thread's q-th load
  __device__ static uint32_t voff(int q, int ld, int rows) {
    const int p = (q * (NT / 64) + (int)threadIdx.x / 64) * 64 + (int)threadIdx.x % 64;
    const int r = p / CPR, kc = (p % CPR) ^ swz<HD>(r);
    return 2u * (uint32_t)(min(r, rows - 1) * ld + kc * 8);
  }
  // the tile's rows [row0, row0 + KB) of g (rows below S valid) into the LDS tile at lds
  __device__ static void issue(const bf16* g, int ld, int row0, int S, uint32_t lds) {
    const bf16* t = g + (int64_t)row0 * ld;
    const uint32_t w = (uint32_t)__builtin_amdgcn_readfirstlane(threadIdx.x / 64) * 1024u;
#pragma unroll
    for (int q = 0; q < PER; ++q) dma16(t, voff(q, ld, S - row0), lds + w + (uint32_t)q * (NT / 64) * 1024u);
  }
};

// stages of the streamed-tile ring: a tile's loads are issued NS - 1 iterations before it is used
template <int HD>
constexpr int ring_stages() { return HD == 64 ? 3 : 2; }

// Waits until this thread's loads of the current iteration's stage are in LDS: issued after them
// are the loads of the next NS - 2 iterations, those that exist (`more` = the next iteration does)
template <int NS, int PER_STAGE>
__device__ __forceinline__ void ring_wait(bool more) {
  if constexpr (NS >= 3) {
    if (more) wait_vm_lds<(NS - 2) * PER_STAGE>();
    else wait_vm_lds<0>();
  } else {
    wait_vm_lds<0>();
  }
}

// Writes a wave's 32 columns of X^T (accumulators: rows d, column = the wave's 32 rows) as rows of
// out (row stride ldo) through the LDS staging area, scaled.  Ends with all staging reads done.
// With rope tables the rows are gradients w.r.t. RoPE-rotated vectors and leave rotated back by
// -angle(position, i) (position = row within the sequence): the gradient w.r.t. the unrotated ones.
template <int HD>
__device__ __forceinline__ void store_rows_from_t(float* __restrict__ stage, const f32x16* acc, float scale,
                                                  bf16* __restrict__ out, int ldo, int row0_wg, int S,
                                                  const float* rope_cos = nullptr,
                                                  const float* rope_sin = nullptr,
                                                  float* __restrict__ out32 = nullptr) {
  constexpr int OP = HD + 4;  // fp32 staging pitch
  const int wave = threadIdx.x / 64, lane = threadIdx.x % 64, half = lane / 32, col = lane % 32;
#pragma unroll
  for (int dt = 0; dt < HD / 32; ++dt)
#pragma unroll
    for (int e = 0; e < 16; ++e)
      stage[(wave * 32 + col) * OP + dt * 32 + 8 * (e / 4) + 4 * half + (e % 4)] = acc[dt][e] * scale;
  __syncthreads();
  for (int c = threadIdx.x; c < QB * HD / 8; c += NT) {
    const int r = c / (HD / 8), d = (c % (HD / 8)) * 8;
    const int row = row0_wg + r;
    if (row >= S) continue;
    const float* sr = stage + r * OP;
    bf16x8 ov;
    if (rope_cos) {
      constexpr int HH = HD / 2;
      const bool first = d < HH;
      const int i0 = d % HH;
      const float* xp = sr + (first ? d + HH : d - HH);
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        const float cs = rope_cos[row * HH + i0 + q], sn = rope_sin[row * HH + i0 + q];
        ov[q] = (bf16)(first ? sr[d + q] * cs + xp[q] * sn : sr[d + q] * cs - xp[q] * sn);
      }
    } else {
#pragma unroll
      for (int q = 0; q < 8; ++q) ov[q] = (bf16)sr[d + q];
      if (out32) {  // the fp32 rows too (same layout)
        float* o32 = out32 + (int64_t)row * ldo + d;
        *reinterpret_cast<f32x4*>(o32) = f32x4{sr[d], sr[d + 1], sr[d + 2], sr[d + 3]};
        *reinterpret_cast<f32x4*>(o32 + 4) = f32x4{sr[d + 4], sr[d + 5], sr[d + 6], sr[d + 7]};
      }
    }
    *reinterpret_cast<bf16x8*>(out + (int64_t)row * ldo + d) = ov;
  }
  __syncthreads();
}

// Work item of block L in a 1-D grid of N blocks made of units of per_unit items (a unit: the
// blocks of one head, which stream the same K/V or Q/dO rows).  The hardware places block L on XCD
// L mod 8; when N is a multiple of 8, XCD x gets the contiguous run [x N/8, (x+1) N/8) of items, so
// a unit's blocks share that XCD's L2 instead of each XCD fetching every head.
__device__ __forceinline__ void xcd_item(int L, int N, int per_unit, int& unit, int& idx) {
  const int r = (N % 8 == 0) ? (L % 8) * (N / 8) + L / 8 : L;
  unit = r / per_unit;
  idx = r % per_unit;
}

template <int HD>
struct Lds {
  static constexpr int NS = ring_stages<HD>();
  static constexpr int TSZ = KB * HD;  // elements of one [KB][HD] tile
  static constexpr size_t out_bytes = (size_t)QB * (HD + 4) * 4;  // fp32 output staging
  // forward and dQ: a stage holds a K and a V tile; dK/dV: a Q and a dO tile, then the lse and
  // delta values of the tile's rows
  static constexpr size_t kv_stage = (size_t)2 * TSZ * 2;
  static constexpr size_t qd_stage = (size_t)2 * TSZ * 2 + 2 * KB * 4;
  static constexpr size_t mx(size_t x, size_t y) { return x > y ? x : y; }
  static constexpr size_t fwd_bytes() { return mx(NS * kv_stage, out_bytes); }
  static constexpr size_t dq_bytes() { return fwd_bytes(); }
  static constexpr size_t dkv_bytes() { return mx(NS * qd_stage, out_bytes); }
};

// ------------------------------------------------------------------------------------------ forward
// HILO (a stage that keeps O in fp32 for the backward's delta): P enters the P V product as its
// hi / lo bf16 pair, so that O, and the fp32 copy written to o32, carry P to about 2^-17 instead of
// bf16's 2^-9; delta = rowsum(dO O) is then consistent with the P and dP the backward recomputes.
template <int HD, bool HILO>
__global__ void __launch_bounds__(NT) flash_fwd(AttnArgs a) {
  using L = Lds<HD>;
  using TT = DmaRowTile<HD>;
  constexpr int KS = HD / 16, DT = HD / 32, NS = L::NS;
  extern __shared__ __align__(16) unsigned char smem[];
  bf16* ring = reinterpret_cast<bf16*>(smem);  // [NS][K tile | V tile], swizzled

  const int nqb = (a.S + QB - 1) / QB;
  int unit, idx;  // unit: (batch, query head); heaviest query blocks first
  xcd_item(blockIdx.x, nqb * a.Hq * a.B, nqb, unit, idx);
  const int qb = nqb - 1 - idx;
  const int h = unit % a.Hq, b = unit / a.Hq;
  const int kvh = h / (a.Hq / a.Hkv);
  const int ld = (a.Hq + 2 * a.Hkv) * HD;
  const bf16* base = (const bf16*)a.qkv + (int64_t)b * a.S * ld;
  const bf16* kbase = base + (a.Hq + kvh) * HD;
  const bf16* vbase = base + (a.Hq + a.Hkv + kvh) * HD;
  const int wave = threadIdx.x / 64, lane = threadIdx.x % 64, half = lane / 32, col = lane % 32;
  const int q0 = qb * QB + wave * 32, myq = q0 + col;
  const int nkb = min(a.S - 1, qb * QB + QB - 1) / KB + 1;
  auto issue = [&](int kb) {
    bf16* st = ring + (kb % NS) * 2 * L::TSZ;
    TT::issue(kbase, ld, kb * KB, a.S, lds_addr(st));
    TT::issue(vbase, ld, kb * KB, a.S, lds_addr(st + L::TSZ));
  };
  bf16x8 qf[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    if (myq < a.S) qf[ks] = *reinterpret_cast<const bf16x8*>(base + (int64_t)myq * ld + h * HD + ks * 16 + 8 * half);
    else for (int j = 0; j < 8; ++j) qf[ks][j] = (bf16)0.f;
  }
  // The register loads complete here, so that no wait the compiler places for them lands inside
  // the loop (a vmcnt wait there would also drain the ring's loads in flight).
  wait_vm_lds<0>();
#pragma unroll
  for (int s = 0; s < NS - 1; ++s)
    if (s < nkb) issue(s);
  const float sl2 = LOG2E / sqrtf((float)HD);
  f32x16 o[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
#pragma unroll
    for (int e = 0; e < 16; ++e) o[dt][e] = 0.f;
  float m = -INFINITY, lsum = 0.f;

  for (int kb = 0; kb < nkb; ++kb) {
    ring_wait<NS, 2 * TT::PER>(kb + 1 < nkb);
    block_barrier();  // every thread's loads of tile kb are in; every wave is done with tile kb - 1
    if (kb + NS - 1 < nkb) issue(kb + NS - 1);  // into the stage tile kb - 1 occupied
    const bf16* Ks = ring + (kb % NS) * 2 * L::TSZ;
    const bf16* Vs = Ks + L::TSZ;
    const int key0 = kb * KB;
    if (key0 <= q0 + 31) {  // some key of this block is visible to some query of this wave
      // the two sub-tiles' score chains interleaved, the K fragments of the next 16-deep step
      // read while this step's MFMAs run
      f32x16 s[2];
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int e = 0; e < 16; ++e) s[t][e] = 0.f;
      bf16x8 fk[2][2];
#pragma unroll
      for (int t = 0; t < 2; ++t) fk[0][t] = frag_rows<HD>(Ks, t * 32, 0);
      static_for<KS>([&](auto KSI) {
        constexpr int ks = KSI, c = ks & 1;
        __builtin_amdgcn_sched_barrier(0);
        if constexpr (ks + 1 < KS) {
#pragma unroll
          for (int t = 0; t < 2; ++t) fk[c ^ 1][t] = frag_rows<HD>(Ks, t * 32, (ks + 1) * 16);
        }
#pragma unroll
        for (int t = 0; t < 2; ++t) s[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fk[c][t], qf[ks], s[t], 0, 0, 0);
        if constexpr (ks + 1 < KS) {
          static_for<2>([&](auto) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // one LDS read
          });
        }
        __builtin_amdgcn_sched_barrier(0);
      });
      // row maximum of the raw scores (the scale is positive), masked on the diagonal block
      float bm = -INFINITY;
      if (key0 + KB - 1 > q0) {
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
          for (int e = 0; e < 16; ++e)
            if (key0 + t * 32 + 8 * (e / 4) + 4 * half + (e % 4) > myq) s[t][e] = -INFINITY;
      }
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int e = 0; e < 16; ++e) bm = fmaxf(bm, s[t][e]);
      bm = pair_max(bm) * sl2;  // every query of the wave sees key0 here, so bm is finite
      // Lazy maximum: m (log2 units) moves only when a score exceeds it by more than 8, so
      // p = 2^(s sl2 - m) <= 256 and O is rescaled only when some row's maximum jumps; O / l and
      // lse = m + log2(l) do not depend on which m was used.
      const bool move = bm > m + 8.0f;
      const float mn = move ? bm : m;
      const float corr = (m == -INFINITY) ? 0.f : fast_exp2(m - mn);  // 1 when m stays
      float rs = 0.f;
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const float p = fast_exp2(__builtin_fmaf(s[t][e], sl2, -mn));
          s[t][e] = p;
          rs += p;
        }
      rs = pair_sum(rs);
      lsum = lsum * corr + rs;
      m = mn;
      if (__any(move)) {  // some query of the wave moved its maximum
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
          for (int e = 0; e < 16; ++e) o[dt][e] *= corr;
      }
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        if constexpr (HILO) {
          bf16x8 ph, pl, vfr[DT];
          if (kk % 2) acc_rows_to_b_split<8>(s[kk / 2], ph, pl);
          else acc_rows_to_b_split<0>(s[kk / 2], ph, pl);
#pragma unroll
          for (int dt = 0; dt < DT; ++dt) vfr[dt] = frag_cols<HD>(Vs, dt * 32, kk * 16);
#pragma unroll
          for (int dt = 0; dt < DT; ++dt) o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vfr[dt], ph, o[dt], 0, 0, 0);
#pragma unroll
          for (int dt = 0; dt < DT; ++dt) o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vfr[dt], pl, o[dt], 0, 0, 0);
        } else {
          const bf16x8 pf = (kk % 2) ? acc_rows_to_b<8>(s[kk / 2]) : acc_rows_to_b<0>(s[kk / 2]);
#pragma unroll
          for (int dt = 0; dt < DT; ++dt)
            o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(frag_cols<HD>(Vs, dt * 32, kk * 16), pf, o[dt], 0, 0, 0);
        }
      }
    }
  }
  block_barrier();  // every wave is done with the last tile: the ring becomes the output staging
  if (half == 0 && myq < a.S)
    a.lse[((int64_t)b * a.Hq + h) * a.S + myq] = (m + log2f(lsum)) * 0.6931471805599453f;
  const float inv = lsum > 0.f ? 1.0f / lsum : 0.f;
  store_rows_from_t<HD>(reinterpret_cast<float*>(smem), o, inv,
                        (bf16*)a.o + (int64_t)b * a.S * a.Hq * HD + h * HD, a.Hq * HD, qb * QB, a.S, nullptr,
                        nullptr, HILO ? a.o32 + (int64_t)b * a.S * a.Hq * HD + h * HD : nullptr);
}

// ------------------------------------------------------------------------------------------ dQ
// delta_i = rowsum(dO O)_i comes with the backward's arguments, from O in fp32 (see flash_fwd's
// HILO), so that every row of dS = P (dP - delta) sums to zero with the P and dP recomputed here.
template <int HD>
__device__ __forceinline__ void bwd_dq_block(const AttnArgs& a, int bx, int by, int bz,
    unsigned char* __restrict__ smem) {
  using L = Lds<HD>;
  using TT = DmaRowTile<HD>;
  constexpr int KS = HD / 16, DT = HD / 32, NS = L::NS;
  bf16* ring = reinterpret_cast<bf16*>(smem);  // [NS][K tile | V tile], swizzled
  const int nqb = (a.S + QB - 1) / QB;
  const int qb = nqb - 1 - bx;
  const int h = by, b = bz;
  const int kvh = h / (a.Hq / a.Hkv);
  const int ld = (a.Hq + 2 * a.Hkv) * HD, hqd = a.Hq * HD;
  const bf16* base = (const bf16*)a.qkv + (int64_t)b * a.S * ld;
  const bf16* kbase = base + (a.Hq + kvh) * HD;
  const bf16* vbase = base + (a.Hq + a.Hkv + kvh) * HD;
  const bf16* dob = (const bf16*)a.dout + (int64_t)b * a.S * hqd + h * HD;
  const int wave = threadIdx.x / 64, lane = threadIdx.x % 64, half = lane / 32, col = lane % 32;
  const int q0 = qb * QB + wave * 32, myq = q0 + col;
  const int nkb = min(a.S - 1, qb * QB + QB - 1) / KB + 1;
  auto issue = [&](int kb) {
    bf16* st = ring + (kb % NS) * 2 * L::TSZ;
    TT::issue(kbase, ld, kb * KB, a.S, lds_addr(st));
    TT::issue(vbase, ld, kb * KB, a.S, lds_addr(st + L::TSZ));
  };
  bf16x8 qf[KS], df[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    if (myq < a.S) {
      qf[ks] = *reinterpret_cast<const bf16x8*>(base + (int64_t)myq * ld + h * HD + ks * 16 + 8 * half);
      df[ks] = *reinterpret_cast<const bf16x8*>(dob + (int64_t)myq * hqd + ks * 16 + 8 * half);
    } else {
      for (int j = 0; j < 8; ++j) { qf[ks][j] = (bf16)0.f; df[ks][j] = (bf16)0.f; }
    }
  }
  const int64_t sidx = ((int64_t)b * a.Hq + h) * a.S + min(myq, a.S - 1);
  const float lse2 = a.lse[sidx] * LOG2E, dl = a.delta[sidx];
  wait_vm_lds<0>();  // register loads done before the ring starts (as in the forward)
#pragma unroll
  for (int s = 0; s < NS - 1; ++s)
    if (s < nkb) issue(s);
  const float sl2 = LOG2E / sqrtf((float)HD);
  f32x16 dq[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
#pragma unroll
    for (int e = 0; e < 16; ++e) dq[dt][e] = 0.f;
  for (int kb = 0; kb < nkb; ++kb) {
    ring_wait<NS, 2 * TT::PER>(kb + 1 < nkb);
    block_barrier();  // every thread's loads of tile kb are in; every wave is done with tile kb - 1
    if (kb + NS - 1 < nkb) issue(kb + NS - 1);
    const bf16* Ks = ring + (kb % NS) * 2 * L::TSZ;
    const bf16* Vs = Ks + L::TSZ;
    const int key0 = kb * KB;
    if (key0 <= q0 + 31) {
      // S and dP of both 32-key sub-tiles first, so that the softmax of the first runs on the
      // vector ALUs while the matrix cores work on the second, and the dQ products of the first
      // while the softmax of the second runs
      f32x16 s[2], dp[2];
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int e = 0; e < 16; ++e) { s[t][e] = 0.f; dp[t][e] = 0.f; }
      if constexpr (HD == 128) {
        // the two sub-tiles' four accumulator chains interleaved, the K and V fragments of the
        // next 16-deep step read while this step's MFMAs run
        bf16x8 fk[2][2], fv[2][2];
#pragma unroll
        for (int t = 0; t < 2; ++t) {
          fk[0][t] = frag_rows<HD>(Ks, t * 32, 0);
          fv[0][t] = frag_rows<HD>(Vs, t * 32, 0);
        }
        static_for<KS>([&](auto KSI) {
          constexpr int ks = KSI, c = ks & 1;
          __builtin_amdgcn_sched_barrier(0);
          if constexpr (ks + 1 < KS) {
#pragma unroll
            for (int t = 0; t < 2; ++t) {
              fk[c ^ 1][t] = frag_rows<HD>(Ks, t * 32, (ks + 1) * 16);
              fv[c ^ 1][t] = frag_rows<HD>(Vs, t * 32, (ks + 1) * 16);
            }
          }
#pragma unroll
          for (int t = 0; t < 2; ++t) {
            s[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fk[c][t], qf[ks], s[t], 0, 0, 0);
            dp[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fv[c][t], df[ks], dp[t], 0, 0, 0);
          }
          if constexpr (ks + 1 < KS) {
            static_for<4>([&](auto) {
              __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
              __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // one LDS read
            });
          }
          __builtin_amdgcn_sched_barrier(0);
        });
      } else {
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
          for (int ks = 0; ks < KS; ++ks) {
            s[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(frag_rows<HD>(Ks, t * 32, ks * 16), qf[ks], s[t], 0, 0, 0);
            dp[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(frag_rows<HD>(Vs, t * 32, ks * 16), df[ks], dp[t], 0, 0, 0);
          }
      }
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        // at head dim 128 the K fragments of the sub-tile's dQ products (two transposing reads
        // each) go through a ring of 4, read 3 products ahead, the first three before the softmax
        constexpr int NC = 2 * DT, RA = 3;
        bf16x8 fc[RA + 1];
        if constexpr (HD == 128) {
          static_for<RA>([&](auto QI) {
            constexpr int q = QI;
            fc[q] = frag_cols<HD>(Ks, (q % DT) * 32, t * 32 + (q / DT) * 16);
          });
          __builtin_amdgcn_sched_barrier(0);
        }
        // every key of the sub-tile is visible to every query: no mask (head dim 64 only; at 128
        // the second code path costs the kernel its spill-free register budget)
        if (HD == 64 && key0 + t * 32 + 31 <= q0) {
#pragma unroll
          for (int e = 0; e < 16; ++e) s[t][e] = fast_exp2(__builtin_fmaf(s[t][e], sl2, -lse2)) * (dp[t][e] - dl);
        } else {
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            const int key = key0 + t * 32 + 8 * (e / 4) + 4 * half + (e % 4);
            const float p = key <= myq ? fast_exp2(__builtin_fmaf(s[t][e], sl2, -lse2)) : 0.f;
            s[t][e] = p * (dp[t][e] - dl);
          }
        }
        if constexpr (HD == 128) {
          const bf16x8 b0 = acc_rows_to_b<0>(s[t]), b1 = acc_rows_to_b<8>(s[t]);
          static_for<NC>([&](auto QI) {
            constexpr int q = QI, g2 = q / DT, dt = q % DT;
            __builtin_amdgcn_sched_barrier(0);
            if constexpr (q + RA < NC)
              fc[(q + RA) % (RA + 1)] = frag_cols<HD>(Ks, ((q + RA) % DT) * 32, t * 32 + ((q + RA) / DT) * 16);
            dq[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fc[q % (RA + 1)], g2 ? b1 : b0, dq[dt], 0, 0, 0);
            __builtin_amdgcn_sched_barrier(0);
          });
        } else {
#pragma unroll
          for (int g2 = 0; g2 < 2; ++g2) {
            const bf16x8 bop = g2 ? acc_rows_to_b<8>(s[t]) : acc_rows_to_b<0>(s[t]);
#pragma unroll
            for (int dt = 0; dt < DT; ++dt)
              dq[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(frag_cols<HD>(Ks, dt * 32, t * 32 + g2 * 16), bop, dq[dt], 0, 0, 0);
          }
        }
      }
    }
  }
  block_barrier();  // every wave is done with the last tile: the ring becomes the output staging
  store_rows_from_t<HD>(reinterpret_cast<float*>(smem), dq, 1.0f / sqrtf((float)HD),
                        (bf16*)a.dqkv + (int64_t)b * a.S * ld + h * HD, ld, qb * QB, a.S, a.rope_cos, a.rope_sin);
}

template <int HD>
__global__ void __launch_bounds__(NT) flash_bwd_dq(AttnArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int nqb = (a.S + QB - 1) / QB;
  int unit, idx;  // unit: (batch, query head)
  xcd_item(blockIdx.x, nqb * a.Hq * a.B, nqb, unit, idx);
  bwd_dq_block<HD>(a, idx, unit % a.Hq, unit / a.Hq, smem);
}

// ------------------------------------------------------------------------------------------ dK, dV
template <int HD>
__device__ __forceinline__ void bwd_dkv_block(const AttnArgs& a, int bx, int by, int bz,
    unsigned char* __restrict__ smem) {
  using L = Lds<HD>;
  using TT = DmaRowTile<HD>;
  constexpr int KS = HD / 16, DT = HD / 32, NS = L::NS;
  // stage: Q tile, dO tile (swizzled [KB][HD] each), lse[KB], delta[KB]
  constexpr int SSZ = (int)(L::qd_stage / 2);  // stage size in bf16 elements
  bf16* ring = reinterpret_cast<bf16*>(smem);
  const int kbk = bx;  // block of 128 keys; low blocks see the most queries and go first
  const int kvh = by, b = bz;
  const int group = a.Hq / a.Hkv;
  const int ld = (a.Hq + 2 * a.Hkv) * HD, hqd = a.Hq * HD;
  const bf16* base = (const bf16*)a.qkv + (int64_t)b * a.S * ld;
  const bf16* dbase = (const bf16*)a.dout + (int64_t)b * a.S * hqd;
  const int wave = threadIdx.x / 64, lane = threadIdx.x % 64, half = lane / 32, col = lane % 32;
  const int k0 = kbk * QB + wave * 32, mykey = k0 + col;
  // iterations: every (query head of the group, query block at or after this key block)
  const int qblk0 = (kbk * QB) / KB;
  const int nqblk = (a.S + KB - 1) / KB;
  const int per_head = nqblk - qblk0;
  const int nit = group * per_head;
  // each wave loads one row vector per stage: waves 0 and 2 the lse values, 1 and 3 the deltas
  // (the same data twice, so that every thread has the same number of loads in flight)
  const float* rowv = (__builtin_amdgcn_readfirstlane(wave) & 1) ? a.delta : a.lse;
  auto issue = [&](int it) {
    const int h = kvh * group + it / per_head, qs0 = (qblk0 + it % per_head) * KB;
    bf16* st = ring + (it % NS) * SSZ;
    TT::issue(base + h * HD, ld, qs0, a.S, lds_addr(st));
    TT::issue(dbase + h * HD, hqd, qs0, a.S, lds_addr(st + L::TSZ));
    const float* rv = rowv + ((int64_t)b * a.Hq + h) * a.S;
    dma4(rv, 4u * (uint32_t)min(qs0 + lane, a.S - 1),
         lds_addr(reinterpret_cast<float*>(st + 2 * L::TSZ) + (__builtin_amdgcn_readfirstlane(wave) & 1) * KB));
  };
  bf16x8 kf[KS], vf[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    if (mykey < a.S) {
      kf[ks] = *reinterpret_cast<const bf16x8*>(base + (int64_t)mykey * ld + (a.Hq + kvh) * HD + ks * 16 + 8 * half);
      vf[ks] = *reinterpret_cast<const bf16x8*>(base + (int64_t)mykey * ld + (a.Hq + a.Hkv + kvh) * HD + ks * 16 + 8 * half);
    } else {
      for (int j = 0; j < 8; ++j) { kf[ks][j] = (bf16)0.f; vf[ks][j] = (bf16)0.f; }
    }
  }
  wait_vm_lds<0>();  // register loads done before the ring starts (as in the forward)
#pragma unroll
  for (int s = 0; s < NS - 1; ++s)
    if (s < nit) issue(s);
  const float sl2 = LOG2E / sqrtf((float)HD);
  f32x16 dk[DT], dv[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
#pragma unroll
    for (int e = 0; e < 16; ++e) { dk[dt][e] = 0.f; dv[dt][e] = 0.f; }
  for (int it = 0; it < nit; ++it) {
    ring_wait<NS, 2 * TT::PER + 1>(it + 1 < nit);
    block_barrier();  // every thread's loads of iteration it are in; every wave is done with it - 1
    if (it + NS - 1 < nit) issue(it + NS - 1);
    const bf16* Qs = ring + (it % NS) * SSZ;
    const bf16* Ds = Qs + L::TSZ;
    const float* Ls = reinterpret_cast<const float*>(Qs + 2 * L::TSZ);
    const float* Dl = Ls + KB;
    const int qs0 = (qblk0 + it % per_head) * KB;
    if constexpr (HD == 128) {
      // Both 32-query sub-tiles at once (one wave per SIMD at this head dim, so the wave's own
      // instruction-level parallelism is what hides latency): the S and dP products of the two
      // sub-tiles interleaved (four independent accumulator chains), then the softmax of each
      // sub-tile beside the other's MFMAs.  A sub-tile whose queries all precede the wave's keys
      // gets P = 0 from the causal mask, so it needs no branch.
      f32x16 s2[2], dp2[2];
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int e = 0; e < 16; ++e) { s2[t][e] = 0.f; dp2[t][e] = 0.f; }
      // the Q and dO fragments of the next 16-deep step are read while this step's MFMAs run
      bf16x8 fq[2][2], fd[2][2];
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        fq[0][t] = frag_rows<HD>(Qs, t * 32, 0);
        fd[0][t] = frag_rows<HD>(Ds, t * 32, 0);
      }
      static_for<KS>([&](auto KSI) {
        constexpr int ks = KSI, c = ks & 1;
        __builtin_amdgcn_sched_barrier(0);
        if constexpr (ks + 1 < KS) {
#pragma unroll
          for (int t = 0; t < 2; ++t) {
            fq[c ^ 1][t] = frag_rows<HD>(Qs, t * 32, (ks + 1) * 16);
            fd[c ^ 1][t] = frag_rows<HD>(Ds, t * 32, (ks + 1) * 16);
          }
        }
#pragma unroll
        for (int t = 0; t < 2; ++t) {
          s2[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fq[c][t], kf[ks], s2[t], 0, 0, 0);
          dp2[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fd[c][t], vf[ks], dp2[t], 0, 0, 0);
        }
        if constexpr (ks + 1 < KS) {
          static_for<4>([&](auto) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // one LDS read
          });
        }
        __builtin_amdgcn_sched_barrier(0);
      });
      // dV and dK of each sub-tile: 16 MFMAs, (g2, dt, dV or dK), whose dO or Q fragments (two
      // transposing reads each) stream through a ring of 4 read 3 MFMAs ahead; the first three
      // go out before the sub-tile's softmax
      constexpr int NC = 2 * DT * 2, RA = 3;
      auto cfrag = [&](auto QI, int t) {
        constexpr int q = QI, g2 = q / (2 * DT), dt = (q / 2) % DT, isk = q % 2;
        return frag_cols<HD>(isk ? Qs : Ds, dt * 32, t * 32 + g2 * 16);
      };
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        bf16x8 fc[RA + 1];
        static_for<RA>([&](auto QI) { fc[(int)QI] = cfrag(QI, t); });
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int e4 = 0; e4 < 4; ++e4) {
          const int r0 = t * 32 + 8 * e4 + 4 * half;
          const f32x4 l4 = *reinterpret_cast<const f32x4*>(Ls + r0);
          const f32x4 d4 = *reinterpret_cast<const f32x4*>(Dl + r0);
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const int e = 4 * e4 + j, q = qs0 + r0 + j;
            const float p = (q >= mykey && q < a.S) ? fast_exp2(__builtin_fmaf(s2[t][e], sl2, -l4[j] * LOG2E)) : 0.f;
            s2[t][e] = p;
            dp2[t][e] = p * (dp2[t][e] - d4[j]);
          }
        }
        const bf16x8 pb0 = acc_rows_to_b<0>(s2[t]), pb1 = acc_rows_to_b<8>(s2[t]);
        const bf16x8 sb0 = acc_rows_to_b<0>(dp2[t]), sb1 = acc_rows_to_b<8>(dp2[t]);
        static_for<NC>([&](auto QI) {
          constexpr int q = QI, g2 = q / (2 * DT), dt = (q / 2) % DT, isk = q % 2;
          __builtin_amdgcn_sched_barrier(0);
          if constexpr (q + RA < NC) fc[(q + RA) % (RA + 1)] = cfrag(std::integral_constant<int, q + RA>{}, t);
          if constexpr (isk)
            dk[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fc[q % (RA + 1)], g2 ? sb1 : sb0, dk[dt], 0, 0, 0);
          else
            dv[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fc[q % (RA + 1)], g2 ? pb1 : pb0, dv[dt], 0, 0, 0);
          __builtin_amdgcn_sched_barrier(0);
        });
      }
    } else {
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const int q0t = qs0 + t * 32;
        if (q0t + 31 < k0) continue;  // every query of this sub-tile precedes every key of the wave
        f32x16 s, dp;
#pragma unroll
        for (int e = 0; e < 16; ++e) { s[e] = 0.f; dp[e] = 0.f; }
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(frag_rows<HD>(Qs, t * 32, ks * 16), kf[ks], s, 0, 0, 0);
          dp = __builtin_amdgcn_mfma_f32_32x32x16_bf16(frag_rows<HD>(Ds, t * 32, ks * 16), vf[ks], dp, 0, 0, 0);
        }
        // accumulator rows of this lane: t*32 + 8 (e/4) + 4 half + (e mod 4): four runs of 4
        // consecutive query rows, so lse and delta arrive as 16-byte reads
        // every query of the sub-tile sees every key of the wave and exists: no mask (head dim 64
        // only, as in the dQ kernel)
        const bool full = HD == 64 && q0t >= k0 + 31 && q0t + 31 < a.S;
#pragma unroll
        for (int e4 = 0; e4 < 4; ++e4) {
          const int r0 = t * 32 + 8 * e4 + 4 * half;
          const f32x4 l4 = *reinterpret_cast<const f32x4*>(Ls + r0);
          const f32x4 d4 = *reinterpret_cast<const f32x4*>(Dl + r0);
          if (full) {
#pragma unroll
            for (int j = 0; j < 4; ++j) {
              const int e = 4 * e4 + j;
              const float p = fast_exp2(__builtin_fmaf(s[e], sl2, -l4[j] * LOG2E));
              s[e] = p;
              dp[e] = p * (dp[e] - d4[j]);
            }
          } else {
#pragma unroll
            for (int j = 0; j < 4; ++j) {
              const int e = 4 * e4 + j, q = qs0 + r0 + j;
              const float p = (q >= mykey && q < a.S) ? fast_exp2(__builtin_fmaf(s[e], sl2, -l4[j] * LOG2E)) : 0.f;
              s[e] = p;
              dp[e] = p * (dp[e] - d4[j]);
            }
          }
        }
#pragma unroll
        for (int g2 = 0; g2 < 2; ++g2) {
          const bf16x8 pb = g2 ? acc_rows_to_b<8>(s) : acc_rows_to_b<0>(s);
          const bf16x8 sb = g2 ? acc_rows_to_b<8>(dp) : acc_rows_to_b<0>(dp);
#pragma unroll
          for (int dt = 0; dt < DT; ++dt) {
            dv[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(frag_cols<HD>(Ds, dt * 32, t * 32 + g2 * 16), pb, dv[dt], 0, 0, 0);
            dk[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(frag_cols<HD>(Qs, dt * 32, t * 32 + g2 * 16), sb, dk[dt], 0, 0, 0);
          }
        }
      }
    }
  }
  block_barrier();  // every wave is done with the last stage: the ring becomes the output staging
  bf16* outb = (bf16*)a.dqkv + (int64_t)b * a.S * ld;
  store_rows_from_t<HD>(reinterpret_cast<float*>(smem), dk, 1.0f / sqrtf((float)HD), outb + (a.Hq + kvh) * HD, ld,
                        kbk * QB, a.S, a.rope_cos, a.rope_sin);
  store_rows_from_t<HD>(reinterpret_cast<float*>(smem), dv, 1.0f, outb + (a.Hq + a.Hkv + kvh) * HD, ld, kbk * QB,
                        a.S);
}

template <int HD>
__global__ void __launch_bounds__(NT) flash_bwd_dkv(AttnArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int nkb = (a.S + QB - 1) / QB;
  int unit, idx;  // unit: (batch, key/value head); low key blocks (the most queries) first
  xcd_item(blockIdx.x, nkb * a.Hkv * a.B, nkb, unit, idx);
  bwd_dkv_block<HD>(a, idx, unit % a.Hkv, unit / a.Hkv, smem);
}

// dQ and dK/dV work items in one launch (independent given delta), so the two fill the CUs
// together instead of each leaving a tail.  A unit is one (batch, key/value head): its dK/dV items
// and the dQ items of its query heads, which all stream that head group's rows, on one XCD.
// Within a unit, level k holds dK/dV block k and query block nb - 1 - k of each query head: the
// items of one level have the same causal extent, and heavier levels come first.
template <int HD>
__global__ void __launch_bounds__(NT) flash_bwd_fused(AttnArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int nb = (a.S + QB - 1) / QB;
  const int group = a.Hq / a.Hkv, per_unit = nb * (group + 1);
  int unit, idx;
  xcd_item(blockIdx.x, per_unit * a.Hkv * a.B, per_unit, unit, idx);
  const int kvh = unit % a.Hkv, b = unit / a.Hkv;
  const int level = idx / (group + 1), j = idx % (group + 1);
  if (j == 0) bwd_dkv_block<HD>(a, level, kvh, b, smem);
  else bwd_dq_block<HD>(a, level, kvh * group + j - 1, b, smem);
}

// delta[b, h, i] = sum_d dO[b, i, h, d] O[b, i, h, d]; one thread per (token, head)
template <int HD>
__global__ void __launch_bounds__(256) flash_delta(AttnArgs a) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (int64_t)a.B * a.S * a.Hq) return;
  const int h = idx % a.Hq;
  const int64_t row = idx / a.Hq;  // b * S + i
  const int b = row / a.S, i = row % a.S;
  const bf16* d = (const bf16*)a.dout + row * a.Hq * HD + h * HD;
  float acc = 0.f;
  if (a.o32) {  // O in fp32 (the forward's own copy)
    const float* o = a.o32 + row * a.Hq * HD + h * HD;
#pragma unroll
    for (int c = 0; c < HD; c += 8) {
      const f32x4 x0 = *reinterpret_cast<const f32x4*>(o + c), x1 = *reinterpret_cast<const f32x4*>(o + c + 4);
      const bf16x8 y = *reinterpret_cast<const bf16x8*>(d + c);
#pragma unroll
      for (int j = 0; j < 4; ++j) acc += x0[j] * (float)y[j] + x1[j] * (float)y[j + 4];
    }
  } else {
    const bf16* o = (const bf16*)a.o + row * a.Hq * HD + h * HD;
#pragma unroll
    for (int c = 0; c < HD; c += 8) {
      const bf16x8 x = *reinterpret_cast<const bf16x8*>(o + c);
      const bf16x8 y = *reinterpret_cast<const bf16x8*>(d + c);
#pragma unroll
      for (int j = 0; j < 8; ++j) acc += (float)x[j] * (float)y[j];
    }
  }
  a.delta[((int64_t)b * a.Hq + h) * a.S + i] = acc;
}

template <typename K>
void set_lds(K kernel, size_t bytes) {
  (void)hipFuncSetAttribute((const void*)kernel, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
}

template <int HD, bool HILO>
void fwd_launch(const AttnArgs& a, hipStream_t st) {
  static bool attr = false;
  if (!attr) { set_lds(flash_fwd<HD, HILO>, Lds<HD>::fwd_bytes()); attr = true; }
  flash_fwd<HD, HILO><<<(unsigned)(cdiv(a.S, QB) * a.Hq * a.B), NT, Lds<HD>::fwd_bytes(), st>>>(a);
}

template <int HD>
void bwd_launch(const AttnArgs& a, hipStream_t st) {
  static bool attr = false;
  if (!attr) {
    set_lds(flash_bwd_dq<HD>, Lds<HD>::dq_bytes());
    set_lds(flash_bwd_dkv<HD>, Lds<HD>::dkv_bytes());
    attr = true;
  }
  if (!a.delta_ready) {  // rowsum(dO O), from O in fp32 when the forward kept it
    flash_delta<HD><<<(unsigned)cdiv((int64_t)a.B * a.S * a.Hq, 256), 256, 0, st>>>(a);
  }
  if constexpr (HD == 64) {
    // one launch for both (at head dim 128 the dK/dV register budget would halve dQ's occupancy)
    static bool fattr = false;
    const size_t bytes = std::max(Lds<HD>::dq_bytes(), Lds<HD>::dkv_bytes());
    if (!fattr) { set_lds(flash_bwd_fused<HD>, bytes); fattr = true; }
    const int nb = (int)cdiv(a.S, QB);
    flash_bwd_fused<HD><<<(unsigned)(nb * (a.Hq + a.Hkv) * a.B), NT, bytes, st>>>(a);
  } else {
    flash_bwd_dq<HD><<<(unsigned)(cdiv(a.S, QB) * a.Hq * a.B), NT, Lds<HD>::dq_bytes(), st>>>(a);
    flash_bwd_dkv<HD><<<(unsigned)(cdiv(a.S, QB) * a.Hkv * a.B), NT, Lds<HD>::dkv_bytes(), st>>>(a);
  }
}

}  // namespace

bool attention_mfma_fwd_try(const AttnArgs& a, hipStream_t st) {
  if ((uintptr_t)a.qkv % 16 || (uintptr_t)a.o % 16 || (uintptr_t)a.o32 % 16) return false;
  if (a.o32) {
    if (a.hd == 64) { fwd_launch<64, true>(a, st); return true; }
    if (a.hd == 128) { fwd_launch<128, true>(a, st); return true; }
    return false;
  }
  if (a.hd == 64) { fwd_launch<64, false>(a, st); return true; }
  if (a.hd == 128) { fwd_launch<128, false>(a, st); return true; }
  return false;
}

bool attention_mfma_delta_try(const AttnArgs& a, hipStream_t st) {
  if ((uintptr_t)a.o % 16 || (uintptr_t)a.dout % 16) return false;
  const unsigned nb = (unsigned)cdiv((int64_t)a.B * a.S * a.Hq, 256);
  if (a.hd == 64) { flash_delta<64><<<nb, 256, 0, st>>>(a); return true; }
  if (a.hd == 128) { flash_delta<128><<<nb, 256, 0, st>>>(a); return true; }
  return false;
}

bool attention_mfma_bwd_try(const AttnArgs& a, hipStream_t st) {
  if ((uintptr_t)a.qkv % 16 || (uintptr_t)a.o % 16 || (uintptr_t)a.dout % 16 || (uintptr_t)a.dqkv % 16) return false;
  if (a.hd == 64) { bwd_launch<64>(a, st); return true; }
  if (a.hd == 128) { bwd_launch<128>(a, st); return true; }
  return false;
}
