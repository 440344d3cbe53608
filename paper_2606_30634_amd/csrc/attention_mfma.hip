// Causal grouped-query flash attention on gfx950 matrix cores (bf16 in, fp32 accumulation).
//
// Forward, per (batch, query head, block of 128 queries); each of the 4 waves owns 32 queries and
// walks the key blocks of 64 keys up to its diagonal:
//   S^T = K Q^T            v_mfma_f32_32x32x16_bf16, A = K rows from LDS, B = the wave's Q rows
//                          held in registers; lane l then owns query column l mod 32, so the
//                          softmax statistics of a query live in one lane pair (l, l ^ 32)
//   online softmax         running max m and sum l per query, exp2 with the 1/sqrt(hd) scale and
//                          log2(e) folded into one multiplier
//   O^T += V^T P^T         A = V^T from LDS (V is transposed into [d][key] while staged),
//                          B = P^T rebuilt from the S^T accumulators with one lane-pair exchange
// K and V^T tiles are double-buffered: the next key block is fetched into registers while the
// current one feeds the MFMAs.  O goes out through LDS as 16-byte rows; lse = ln(sum exp(S)) per
// query row is kept for the backward pass.
#include "common.h"
#include "kernels.h"

namespace {

constexpr int QB = 128;   // queries per workgroup
constexpr int KB = 64;    // keys per block
constexpr int NT = 256;   // 4 waves

__device__ __forceinline__ uint32_t lo_pair(uint32_t x, uint32_t y) { return (x & 0xffffu) | (y << 16); }
__device__ __forceinline__ uint32_t hi_pair(uint32_t x, uint32_t y) { return (x >> 16) | (y & 0xffff0000u); }

__device__ __forceinline__ uint32_t pack2(float a, float b) {
  bf16 x = (bf16)a, y = (bf16)b;
  uint16_t u, v;
  __builtin_memcpy(&u, &x, 2);
  __builtin_memcpy(&v, &y, 2);
  return (uint32_t)u | ((uint32_t)v << 16);
}

template <int HD>
struct FwdSmem {
  static constexpr int KP = HD + 8;   // K tile row pitch (elements): [key][d]
  static constexpr int VP = KB + 8;   // V^T tile row pitch: [d][key]
  static constexpr int KSZ = KB * KP;
  static constexpr int VSZ = HD * VP;
  static constexpr int OP = HD + 8;   // output staging pitch: [query][d]
  static constexpr size_t bytes() {
    const size_t kv = (size_t)2 * (KSZ + VSZ) * 2;
    const size_t o = (size_t)QB * OP * 2;
    return kv > o ? kv : o;
  }
};

// K tile: KB keys x HD, 16-byte chunks of 8 d; V tile: chunks of 4 d x 8 keys (8-byte loads along d),
// transposed in registers into [d][key].
template <int HD>
struct KVLoader {
  static constexpr int KCH = KB * HD / 8 / NT;    // K chunks per thread
  static constexpr int VCH = HD * KB / 32 / NT;   // V chunks per thread (may be fractional -> guarded)
  static constexpr int VCHR = VCH > 0 ? VCH : 1;
  uint4 k[KCH];
  uint2 v[VCHR][8];

  __device__ __forceinline__ void load(const bf16* __restrict__ kbase, const bf16* __restrict__ vbase,
                                       int ld, int key0, int S) {
#pragma unroll
    for (int p = 0; p < KCH; ++p) {
      const int c = threadIdx.x + p * NT;
      const int key = key0 + c / (HD / 8), d = (c % (HD / 8)) * 8;
      k[p] = key < S ? *reinterpret_cast<const uint4*>(kbase + (int64_t)key * ld + d) : make_uint4(0u, 0u, 0u, 0u);
    }
#pragma unroll
    for (int p = 0; p < VCHR; ++p) {
      const int c = threadIdx.x + p * NT;
      if (c < HD * KB / 32) {
        const int d = (c % (HD / 4)) * 4, kb = key0 + (c / (HD / 4)) * 8;
#pragma unroll
        for (int j = 0; j < 8; ++j)
          v[p][j] = (kb + j < S) ? *reinterpret_cast<const uint2*>(vbase + (int64_t)(kb + j) * ld + d)
                                 : make_uint2(0u, 0u);
      }
    }
  }
  __device__ __forceinline__ void store(bf16* __restrict__ Ks, bf16* __restrict__ Vt) const {
    using L = FwdSmem<HD>;
#pragma unroll
    for (int p = 0; p < KCH; ++p) {
      const int c = threadIdx.x + p * NT;
      *reinterpret_cast<uint4*>(Ks + (c / (HD / 8)) * L::KP + (c % (HD / 8)) * 8) = k[p];
    }
#pragma unroll
    for (int p = 0; p < VCHR; ++p) {
      const int c = threadIdx.x + p * NT;
      if (c < HD * KB / 32) {
        const int d = (c % (HD / 4)) * 4, kk = (c / (HD / 4)) * 8;
        bf16* base = Vt + d * L::VP + kk;
        uint4 o0, o1, o2, o3;
        o0.x = lo_pair(v[p][0].x, v[p][1].x); o0.y = lo_pair(v[p][2].x, v[p][3].x);
        o0.z = lo_pair(v[p][4].x, v[p][5].x); o0.w = lo_pair(v[p][6].x, v[p][7].x);
        o1.x = hi_pair(v[p][0].x, v[p][1].x); o1.y = hi_pair(v[p][2].x, v[p][3].x);
        o1.z = hi_pair(v[p][4].x, v[p][5].x); o1.w = hi_pair(v[p][6].x, v[p][7].x);
        o2.x = lo_pair(v[p][0].y, v[p][1].y); o2.y = lo_pair(v[p][2].y, v[p][3].y);
        o2.z = lo_pair(v[p][4].y, v[p][5].y); o2.w = lo_pair(v[p][6].y, v[p][7].y);
        o3.x = hi_pair(v[p][0].y, v[p][1].y); o3.y = hi_pair(v[p][2].y, v[p][3].y);
        o3.z = hi_pair(v[p][4].y, v[p][5].y); o3.w = hi_pair(v[p][6].y, v[p][7].y);
        *reinterpret_cast<uint4*>(base) = o0;
        *reinterpret_cast<uint4*>(base + L::VP) = o1;
        *reinterpret_cast<uint4*>(base + 2 * L::VP) = o2;
        *reinterpret_cast<uint4*>(base + 3 * L::VP) = o3;
      }
    }
  }
};

template <int HD>
__global__ void __launch_bounds__(NT) flash_fwd(AttnArgs a) {
  using L = FwdSmem<HD>;
  constexpr int KS = HD / 16;  // k-steps of S^T over the head dimension
  constexpr int DT = HD / 32;  // 32-row tiles of O^T
  extern __shared__ __align__(16) unsigned char smem[];
  bf16* Ks0 = reinterpret_cast<bf16*>(smem);
  bf16* Vt0 = Ks0 + 2 * L::KSZ;

  const int nqb = (a.S + QB - 1) / QB;
  const int qb = nqb - 1 - blockIdx.x;   // heaviest (longest causal range) blocks first
  const int h = blockIdx.y, b = blockIdx.z;
  const int kvh = h / (a.Hq / a.Hkv);
  const int ld = (a.Hq + 2 * a.Hkv) * HD;
  const bf16* base = (const bf16*)a.qkv + (int64_t)b * a.S * ld;
  const bf16* qbase = base + h * HD;
  const bf16* kbase = base + (a.Hq + kvh) * HD;
  const bf16* vbase = base + (a.Hq + a.Hkv + kvh) * HD;

  const int wave = threadIdx.x / 64, lane = threadIdx.x % 64, half = lane / 32, col = lane % 32;
  const int q0 = qb * QB + wave * 32;
  const int myq = q0 + col;

  // this lane's query row as the B operand of S^T = K Q^T (8 consecutive d per k-step)
  bf16x8 qf[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    if (myq < a.S) qf[ks] = *reinterpret_cast<const bf16x8*>(qbase + (int64_t)myq * ld + ks * 16 + 8 * half);
    else for (int j = 0; j < 8; ++j) qf[ks][j] = (bf16)0.f;
  }
  const float sl2 = 1.4426950408889634f / sqrtf((float)HD);  // log2(e) / sqrt(hd)

  f32x16 o[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
#pragma unroll
    for (int e = 0; e < 16; ++e) o[dt][e] = 0.f;
  float m = -INFINITY, lsum = 0.f;

  const int last_key = min(a.S - 1, qb * QB + QB - 1);
  const int nkb = last_key / KB + 1;
  KVLoader<HD> ld_kv;
  ld_kv.load(kbase, vbase, ld, 0, a.S);
  ld_kv.store(Ks0, Vt0);
  __syncthreads();
  for (int kb = 0; kb < nkb; ++kb) {
    const int cur = kb & 1;
    if (kb + 1 < nkb) ld_kv.load(kbase, vbase, ld, (kb + 1) * KB, a.S);
    const bf16* Ks = Ks0 + cur * L::KSZ;
    const bf16* Vt = Vt0 + cur * L::VSZ;
    const int key0 = kb * KB;
    if (key0 <= q0 + 31) {  // some key of this block is visible to some query of this wave
      f32x16 s[2];
#pragma unroll
      for (int t = 0; t < 2; ++t) {
#pragma unroll
        for (int e = 0; e < 16; ++e) s[t][e] = 0.f;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const bf16x8 kf = *reinterpret_cast<const bf16x8*>(Ks + (t * 32 + col) * L::KP + ks * 16 + 8 * half);
          s[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[ks], s[t], 0, 0, 0);
        }
      }
      // scale, causal mask, block max for this query column
      float bm = -INFINITY;
      const bool diag = key0 + KB - 1 > q0;
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          float v = s[t][e] * sl2;
          if (diag) {
            const int key = key0 + t * 32 + 8 * (e / 4) + 4 * half + (e % 4);
            if (key > myq) v = -INFINITY;
          }
          s[t][e] = v;
          bm = fmaxf(bm, v);
        }
      bm = fmaxf(bm, __shfl_xor(bm, 32, 64));
      const float mn = fmaxf(m, bm);
      // a query row whose keys in this block are all masked keeps mn = m (or -inf): guard exp2
      const float corr = (m == -INFINITY) ? 0.f : exp2f(m - mn);
      float rs = 0.f;
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const float p = (s[t][e] == -INFINITY) ? 0.f : exp2f(s[t][e] - mn);
          s[t][e] = p;
          rs += p;
        }
      rs += __shfl_xor(rs, 32, 64);
      lsum = lsum * corr + rs;
      m = mn;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int e = 0; e < 16; ++e) o[dt][e] *= corr;
      // O^T += V^T P^T over the 4 groups of 16 keys
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        const int t = kk / 2, ib = 8 * (kk % 2);
        // own keys of this 16-key group: half 0 holds +0..3 (ib..ib+3), half 1 holds +12..15 (ib+4..ib+7)
        const uint32_t own0 = pack2(s[t][ib + 4 * half + 0], s[t][ib + 4 * half + 1]);
        const uint32_t own1 = pack2(s[t][ib + 4 * half + 2], s[t][ib + 4 * half + 3]);
        const uint32_t snd0 = pack2(s[t][ib + 4 * (1 - half) + 0], s[t][ib + 4 * (1 - half) + 1]);
        const uint32_t snd1 = pack2(s[t][ib + 4 * (1 - half) + 2], s[t][ib + 4 * (1 - half) + 3]);
        const uint32_t rcv0 = __shfl_xor(snd0, 32, 64);
        const uint32_t rcv1 = __shfl_xor(snd1, 32, 64);
        uint32_t pw[4];
        if (half == 0) { pw[0] = own0; pw[1] = own1; pw[2] = rcv0; pw[3] = rcv1; }
        else { pw[0] = rcv0; pw[1] = rcv1; pw[2] = own0; pw[3] = own1; }
        bf16x8 pf;
        __builtin_memcpy(&pf, pw, 16);
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
          const bf16x8 vf = *reinterpret_cast<const bf16x8*>(Vt + (dt * 32 + col) * L::VP + kk * 16 + 8 * half);
          o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf, o[dt], 0, 0, 0);
        }
      }
    }
    if (kb + 1 < nkb) ld_kv.store(Ks0 + (cur ^ 1) * L::KSZ, Vt0 + (cur ^ 1) * L::VSZ);
    __syncthreads();
  }
  // epilogue: O = O^T / l through LDS as [query][d] rows; lse in natural log
  const float inv = lsum > 0.f ? 1.0f / lsum : 0.f;
  bf16* Os = reinterpret_cast<bf16*>(smem);
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int d = dt * 32 + 8 * (e / 4) + 4 * half + (e % 4);
      Os[(wave * 32 + col) * L::OP + d] = (bf16)(o[dt][e] * inv);
    }
  if (half == 0 && myq < a.S)
    a.lse[((int64_t)b * a.Hq + h) * a.S + myq] = (m + log2f(lsum)) * 0.6931471805599453f;
  __syncthreads();
  bf16* out = (bf16*)a.o;
  const int hqd = a.Hq * HD;
  for (int c = threadIdx.x; c < QB * HD / 8; c += NT) {
    const int r = c / (HD / 8), d = (c % (HD / 8)) * 8;
    const int q = qb * QB + r;
    if (q < a.S)
      *reinterpret_cast<uint4*>(out + ((int64_t)b * a.S + q) * hqd + h * HD + d) =
          *reinterpret_cast<const uint4*>(Os + r * L::OP + d);
  }
}

template <int HD>
void fwd_launch(const AttnArgs& a, hipStream_t st) {
  const size_t lds = FwdSmem<HD>::bytes();
  static bool attr = false;
  if (!attr) {
    (void)hipFuncSetAttribute((const void*)flash_fwd<HD>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    attr = true;
  }
  flash_fwd<HD><<<dim3((unsigned)cdiv(a.S, QB), a.Hq, a.B), NT, lds, st>>>(a);
}

bool attention_mfma_fwd_try_impl(const AttnArgs& a, hipStream_t st) {
  if ((uintptr_t)a.qkv % 16 || (uintptr_t)a.o % 16) return false;
  if (a.hd == 64) { fwd_launch<64>(a, st); return true; }
  if (a.hd == 128) { fwd_launch<128>(a, st); return true; }
  return false;
}

// ------------------------------------------------------------------------------------------------
// Backward.  dS = P (dP - delta), delta_i = sum_d dO_id O_id, P = exp(S / sqrt(hd) - lse).
//   dq kernel  (wave owns 32 queries; Q, dO rows in registers):  S^T = K Q^T, dP^T = V dO^T,
//              dQ^T += K^T dS^T                       (A = K, V, K^T tiles from LDS)
//   dkv kernel (wave owns 32 keys; K, V rows in registers; loops over the query heads of its
//              key/value head and the query blocks at or after its keys):  S = Q K^T,
//              dP = dO V^T, dV^T += dO^T P, dK^T += Q^T dS   (A = Q, dO, Q^T, dO^T tiles from LDS)
// No float atomics: every dq, dk, dv element is written by exactly one lane.
// ------------------------------------------------------------------------------------------------

// B operand (8 consecutive k at column lane mod 32) built from a 32x32 accumulator whose rows are
// the k index, for the 16-row group starting at accumulator index ib (0 or 8); one lane-pair swap.
__device__ __forceinline__ bf16x8 acc_rows_to_b(const f32x16& s, int ib, int half) {
  const uint32_t own0 = pack2(s[ib + 4 * half + 0], s[ib + 4 * half + 1]);
  const uint32_t own1 = pack2(s[ib + 4 * half + 2], s[ib + 4 * half + 3]);
  const uint32_t snd0 = pack2(s[ib + 4 * (1 - half) + 0], s[ib + 4 * (1 - half) + 1]);
  const uint32_t snd1 = pack2(s[ib + 4 * (1 - half) + 2], s[ib + 4 * (1 - half) + 3]);
  const uint32_t rcv0 = __shfl_xor(snd0, 32, 64);
  const uint32_t rcv1 = __shfl_xor(snd1, 32, 64);
  uint32_t pw[4];
  if (half == 0) { pw[0] = own0; pw[1] = own1; pw[2] = rcv0; pw[3] = rcv1; }
  else { pw[0] = rcv0; pw[1] = rcv1; pw[2] = own0; pw[3] = own1; }
  bf16x8 r;
  __builtin_memcpy(&r, pw, 16);
  return r;
}

// [R][HD] tile (row pitch P) <- rows row0.. of g (row stride ld); rows >= S are zero
template <int R, int HD, int P>
__device__ __forceinline__ void tile_rows(bf16* __restrict__ dst, const bf16* __restrict__ g, int ld, int row0, int S) {
  for (int c = threadIdx.x; c < R * HD / 8; c += NT) {
    const int r = c / (HD / 8), d = (c % (HD / 8)) * 8;
    const uint4 v = row0 + r < S ? *reinterpret_cast<const uint4*>(g + (int64_t)(row0 + r) * ld + d)
                                 : make_uint4(0u, 0u, 0u, 0u);
    *reinterpret_cast<uint4*>(dst + r * P + d) = v;
  }
}

// [HD][R] tile (row pitch P) <- the transpose of rows row0.. of g; rows >= S are zero
template <int R, int HD, int P>
__device__ __forceinline__ void tile_trans(bf16* __restrict__ dst, const bf16* __restrict__ g, int ld, int row0, int S) {
  for (int c = threadIdx.x; c < HD * R / 32; c += NT) {
    const int d = (c % (HD / 4)) * 4, rb = (c / (HD / 4)) * 8;
    uint2 v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j)
      v[j] = (row0 + rb + j < S) ? *reinterpret_cast<const uint2*>(g + (int64_t)(row0 + rb + j) * ld + d)
                                 : make_uint2(0u, 0u);
    bf16* base = dst + d * P + rb;
    uint4 o0, o1, o2, o3;
    o0.x = lo_pair(v[0].x, v[1].x); o0.y = lo_pair(v[2].x, v[3].x); o0.z = lo_pair(v[4].x, v[5].x); o0.w = lo_pair(v[6].x, v[7].x);
    o1.x = hi_pair(v[0].x, v[1].x); o1.y = hi_pair(v[2].x, v[3].x); o1.z = hi_pair(v[4].x, v[5].x); o1.w = hi_pair(v[6].x, v[7].x);
    o2.x = lo_pair(v[0].y, v[1].y); o2.y = lo_pair(v[2].y, v[3].y); o2.z = lo_pair(v[4].y, v[5].y); o2.w = lo_pair(v[6].y, v[7].y);
    o3.x = hi_pair(v[0].y, v[1].y); o3.y = hi_pair(v[2].y, v[3].y); o3.z = hi_pair(v[4].y, v[5].y); o3.w = hi_pair(v[6].y, v[7].y);
    *reinterpret_cast<uint4*>(base) = o0;
    *reinterpret_cast<uint4*>(base + P) = o1;
    *reinterpret_cast<uint4*>(base + 2 * P) = o2;
    *reinterpret_cast<uint4*>(base + 3 * P) = o3;
  }
}

// Writes a wave's 32 columns of X^T (accumulators: rows d, column = the wave's row c) as rows of
// out (row stride ldo) through the LDS staging area, scaled.
template <int HD>
__device__ __forceinline__ void store_rows_from_t(bf16* __restrict__ stage, const f32x16* acc, float scale,
                                                  bf16* __restrict__ out, int ldo, int row0_wg, int S) {
  constexpr int OP = HD + 8;
  const int wave = threadIdx.x / 64, lane = threadIdx.x % 64, half = lane / 32, col = lane % 32;
#pragma unroll
  for (int dt = 0; dt < HD / 32; ++dt)
#pragma unroll
    for (int e = 0; e < 16; ++e)
      stage[(wave * 32 + col) * OP + dt * 32 + 8 * (e / 4) + 4 * half + (e % 4)] = (bf16)(acc[dt][e] * scale);
  __syncthreads();
  for (int c = threadIdx.x; c < QB * HD / 8; c += NT) {
    const int r = c / (HD / 8), d = (c % (HD / 8)) * 8;
    if (row0_wg + r < S)
      *reinterpret_cast<uint4*>(out + (int64_t)(row0_wg + r) * ldo + d) = *reinterpret_cast<const uint4*>(stage + r * OP + d);
  }
}

template <int HD>
struct BwdSmem {
  static constexpr int RP = HD + 8;  // [row][d] pitch
  static constexpr int TP = KB + 8;  // [d][row] pitch
  static constexpr int RSZ = KB * RP;
  static constexpr int TSZ = HD * TP;
  static constexpr size_t dq_bytes() {
    const size_t t = (size_t)(2 * RSZ + TSZ) * 2, o = (size_t)QB * (HD + 8) * 2;
    return t > o ? t : o;
  }
  static constexpr size_t dkv_bytes() {
    const size_t t = (size_t)(2 * RSZ + 2 * TSZ) * 2 + 2 * KB * 4, o = (size_t)QB * (HD + 8) * 2;
    return t > o ? t : o;
  }
};

template <int HD>
__global__ void __launch_bounds__(NT) flash_bwd_dq(AttnArgs a) {
  using L = BwdSmem<HD>;
  constexpr int KS = HD / 16, DT = HD / 32;
  extern __shared__ __align__(16) unsigned char smem[];
  bf16* Ks = reinterpret_cast<bf16*>(smem);
  bf16* Vs = Ks + L::RSZ;
  bf16* Kt = Vs + L::RSZ;
  const int nqb = (a.S + QB - 1) / QB;
  const int qb = nqb - 1 - blockIdx.x;
  const int h = blockIdx.y, b = blockIdx.z;
  const int kvh = h / (a.Hq / a.Hkv);
  const int ld = (a.Hq + 2 * a.Hkv) * HD, hqd = a.Hq * HD;
  const bf16* base = (const bf16*)a.qkv + (int64_t)b * a.S * ld;
  const bf16* kbase = base + (a.Hq + kvh) * HD;
  const bf16* vbase = base + (a.Hq + a.Hkv + kvh) * HD;
  const bf16* dob = (const bf16*)a.dout + (int64_t)b * a.S * hqd + h * HD;
  const int wave = threadIdx.x / 64, lane = threadIdx.x % 64, half = lane / 32, col = lane % 32;
  const int q0 = qb * QB + wave * 32, myq = q0 + col;
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
  const float lse2 = a.lse[sidx] * 1.4426950408889634f, dl = a.delta[sidx];
  const float sl2 = 1.4426950408889634f / sqrtf((float)HD);
  f32x16 dq[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
#pragma unroll
    for (int e = 0; e < 16; ++e) dq[dt][e] = 0.f;
  const int last_key = min(a.S - 1, qb * QB + QB - 1);
  const int nkb = last_key / KB + 1;
  for (int kb = 0; kb < nkb; ++kb) {
    const int key0 = kb * KB;
    tile_rows<KB, HD, L::RP>(Ks, kbase, ld, key0, a.S);
    tile_rows<KB, HD, L::RP>(Vs, vbase, ld, key0, a.S);
    tile_trans<KB, HD, L::TP>(Kt, kbase, ld, key0, a.S);
    __syncthreads();
    if (key0 <= q0 + 31) {
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        f32x16 s, dp;
#pragma unroll
        for (int e = 0; e < 16; ++e) { s[e] = 0.f; dp[e] = 0.f; }
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const bf16x8 kf = *reinterpret_cast<const bf16x8*>(Ks + (t * 32 + col) * L::RP + ks * 16 + 8 * half);
          const bf16x8 vf = *reinterpret_cast<const bf16x8*>(Vs + (t * 32 + col) * L::RP + ks * 16 + 8 * half);
          s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[ks], s, 0, 0, 0);
          dp = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, df[ks], dp, 0, 0, 0);
        }
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int key = key0 + t * 32 + 8 * (e / 4) + 4 * half + (e % 4);
          const float p = key <= myq ? exp2f(s[e] * sl2 - lse2) : 0.f;
          s[e] = p * (dp[e] - dl);
        }
#pragma unroll
        for (int g2 = 0; g2 < 2; ++g2) {
          const bf16x8 bop = acc_rows_to_b(s, 8 * g2, half);
#pragma unroll
          for (int dt = 0; dt < DT; ++dt) {
            const bf16x8 kt = *reinterpret_cast<const bf16x8*>(Kt + (dt * 32 + col) * L::TP + t * 32 + g2 * 16 + 8 * half);
            dq[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kt, bop, dq[dt], 0, 0, 0);
          }
        }
      }
    }
    __syncthreads();
  }
  store_rows_from_t<HD>(reinterpret_cast<bf16*>(smem), dq, 1.0f / sqrtf((float)HD),
                        (bf16*)a.dqkv + (int64_t)b * a.S * ld + h * HD, ld, qb * QB, a.S);
}

template <int HD>
__global__ void __launch_bounds__(NT) flash_bwd_dkv(AttnArgs a) {
  using L = BwdSmem<HD>;
  constexpr int KS = HD / 16, DT = HD / 32;
  extern __shared__ __align__(16) unsigned char smem[];
  bf16* Qs = reinterpret_cast<bf16*>(smem);
  bf16* Ds = Qs + L::RSZ;
  bf16* Qt = Ds + L::RSZ;
  bf16* Dt = Qt + L::TSZ;
  float* Ls = reinterpret_cast<float*>(Dt + L::TSZ);
  float* Dl = Ls + KB;
  const int kbk = blockIdx.x;  // block of 128 keys; low blocks see the most queries and go first
  const int kvh = blockIdx.y, b = blockIdx.z;
  const int group = a.Hq / a.Hkv;
  const int ld = (a.Hq + 2 * a.Hkv) * HD, hqd = a.Hq * HD;
  const bf16* base = (const bf16*)a.qkv + (int64_t)b * a.S * ld;
  const int wave = threadIdx.x / 64, lane = threadIdx.x % 64, half = lane / 32, col = lane % 32;
  const int k0 = kbk * QB + wave * 32, mykey = k0 + col;
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
  const float sl2 = 1.4426950408889634f / sqrtf((float)HD);
  f32x16 dk[DT], dv[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
#pragma unroll
    for (int e = 0; e < 16; ++e) { dk[dt][e] = 0.f; dv[dt][e] = 0.f; }
  const int qblk0 = (kbk * QB) / KB;
  const int nqblk = (a.S + KB - 1) / KB;
  for (int hh = 0; hh < group; ++hh) {
    const int h = kvh * group + hh;
    const bf16* qbase = base + h * HD;
    const bf16* dob = (const bf16*)a.dout + (int64_t)b * a.S * hqd + h * HD;
    const int64_t srow = ((int64_t)b * a.Hq + h) * a.S;
    for (int qk = qblk0; qk < nqblk; ++qk) {
      const int qs0 = qk * KB;
      tile_rows<KB, HD, L::RP>(Qs, qbase, ld, qs0, a.S);
      tile_rows<KB, HD, L::RP>(Ds, dob, hqd, qs0, a.S);
      tile_trans<KB, HD, L::TP>(Qt, qbase, ld, qs0, a.S);
      tile_trans<KB, HD, L::TP>(Dt, dob, hqd, qs0, a.S);
      if (threadIdx.x < KB) {
        const int q = min(qs0 + (int)threadIdx.x, a.S - 1);
        Ls[threadIdx.x] = a.lse[srow + q] * 1.4426950408889634f;
        Dl[threadIdx.x] = a.delta[srow + q];
      }
      __syncthreads();
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const int q0t = qs0 + t * 32;
        if (q0t + 31 < k0) continue;  // every query of this sub-tile precedes every key of the wave
        f32x16 s, dp;
#pragma unroll
        for (int e = 0; e < 16; ++e) { s[e] = 0.f; dp[e] = 0.f; }
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const bf16x8 qa = *reinterpret_cast<const bf16x8*>(Qs + (t * 32 + col) * L::RP + ks * 16 + 8 * half);
          const bf16x8 da = *reinterpret_cast<const bf16x8*>(Ds + (t * 32 + col) * L::RP + ks * 16 + 8 * half);
          s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qa, kf[ks], s, 0, 0, 0);
          dp = __builtin_amdgcn_mfma_f32_32x32x16_bf16(da, vf[ks], dp, 0, 0, 0);
        }
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int r = t * 32 + 8 * (e / 4) + 4 * half + (e % 4);  // query row within the block
          const int q = qs0 + r;
          const float p = (q >= mykey && q < a.S) ? exp2f(s[e] * sl2 - Ls[r]) : 0.f;
          s[e] = p;
          dp[e] = p * (dp[e] - Dl[r]);
        }
#pragma unroll
        for (int g2 = 0; g2 < 2; ++g2) {
          const bf16x8 pb = acc_rows_to_b(s, 8 * g2, half);
          const bf16x8 sb = acc_rows_to_b(dp, 8 * g2, half);
#pragma unroll
          for (int dt = 0; dt < DT; ++dt) {
            const int off = (dt * 32 + col) * L::TP + t * 32 + g2 * 16 + 8 * half;
            const bf16x8 dta = *reinterpret_cast<const bf16x8*>(Dt + off);
            const bf16x8 qta = *reinterpret_cast<const bf16x8*>(Qt + off);
            dv[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(dta, pb, dv[dt], 0, 0, 0);
            dk[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qta, sb, dk[dt], 0, 0, 0);
          }
        }
      }
      __syncthreads();
    }
  }
  bf16* stage = reinterpret_cast<bf16*>(smem);
  bf16* outb = (bf16*)a.dqkv + (int64_t)b * a.S * ld;
  store_rows_from_t<HD>(stage, dk, 1.0f / sqrtf((float)HD), outb + (a.Hq + kvh) * HD, ld, kbk * QB, a.S);
  __syncthreads();
  store_rows_from_t<HD>(stage, dv, 1.0f, outb + (a.Hq + a.Hkv + kvh) * HD, ld, kbk * QB, a.S);
}

// delta[b, h, i] = sum_d dO[b, i, h, d] O[b, i, h, d]; one thread per (token, head)
template <int HD>
__global__ void __launch_bounds__(256) flash_delta(AttnArgs a) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (int64_t)a.B * a.S * a.Hq) return;
  const int h = idx % a.Hq;
  const int64_t row = idx / a.Hq;  // b * S + i
  const int b = row / a.S, i = row % a.S;
  const bf16* o = (const bf16*)a.o + row * a.Hq * HD + h * HD;
  const bf16* d = (const bf16*)a.dout + row * a.Hq * HD + h * HD;
  float acc = 0.f;
#pragma unroll
  for (int c = 0; c < HD; c += 8) {
    const bf16x8 x = *reinterpret_cast<const bf16x8*>(o + c);
    const bf16x8 y = *reinterpret_cast<const bf16x8*>(d + c);
#pragma unroll
    for (int j = 0; j < 8; ++j) acc += (float)x[j] * (float)y[j];
  }
  a.delta[((int64_t)b * a.Hq + h) * a.S + i] = acc;
}

template <int HD>
void bwd_launch(const AttnArgs& a, hipStream_t st) {
  const size_t l1 = BwdSmem<HD>::dq_bytes(), l2 = BwdSmem<HD>::dkv_bytes();
  static bool attr = false;
  if (!attr) {
    (void)hipFuncSetAttribute((const void*)flash_bwd_dq<HD>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)l1);
    (void)hipFuncSetAttribute((const void*)flash_bwd_dkv<HD>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)l2);
    attr = true;
  }
  flash_delta<HD><<<(unsigned)cdiv((int64_t)a.B * a.S * a.Hq, 256), 256, 0, st>>>(a);
  flash_bwd_dq<HD><<<dim3((unsigned)cdiv(a.S, QB), a.Hq, a.B), NT, l1, st>>>(a);
  flash_bwd_dkv<HD><<<dim3((unsigned)cdiv(a.S, QB), a.Hkv, a.B), NT, l2, st>>>(a);
}

}  // namespace

bool attention_mfma_fwd_try(const AttnArgs& a, hipStream_t st) { return attention_mfma_fwd_try_impl(a, st); }

bool attention_mfma_bwd_try(const AttnArgs& a, hipStream_t st) {
  if ((uintptr_t)a.qkv % 16 || (uintptr_t)a.o % 16 || (uintptr_t)a.dout % 16 || (uintptr_t)a.dqkv % 16) return false;
  if (a.hd == 64) { bwd_launch<64>(a, st); return true; }
  if (a.hd == 128) { bwd_launch<128>(a, st); return true; }
  return false;
}
