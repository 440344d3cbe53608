// Delayed optimizer update: global gradient norm (two deterministic passes) and the fused,
// HBM-bound AdamW + delay + Error-Feedback pass over the flat fp32 master vector.
//
// Per element, iteration t consuming the gradient g of the previous step (Alg. 1, §2):
//   g <- c g                                  c = min(1, clip / (||g|| + 1e-6))   (App. E.1)
//   m <- b1 m + (1 - b1) g ;  v <- b2 v + (1 - b2) g^2                          (AdamW, §2)
//   u  = lr ( (m / bc1) / (sqrt(v / bc2) + eps) + wd x_t )   bc_i = 1 - b_i^k   (Alg. 2 puts
//                                                             the decay on x_t)
//   x_{t+1} = x_t - u                      standard, or the first update ("t <= 1" of Alg. 1)
//   x_{t+1} = x_t - (1 + lam) u + lam u_prev   Error Feedback (§3.2; lam-scaled form App. A.4)
//   u_prev <- u ;  shadow <- cast(x_{t+1})    compute copy for the next step's forward
// Memory traffic per element (fp32 g, EF, bf16 shadow): x, m, v, u_prev read+write (32 B),
// g read (4 B), shadow write (2 B) = 38 B.  Every access is a 16-byte vector per thread,
// consecutive threads on consecutive addresses.
#include "common.h"
#include "kernels.h"

namespace {

constexpr int NORM_BLOCKS = 1024;
constexpr int NORM_THREADS = 256;

// Streaming accesses: every byte of the pass is touched once, so loads and stores are
// non-temporal (they bypass the caches' retention policy) and use native 16- / 8-byte vectors.
template <typename G>
__device__ __forceinline__ void load4(const G* p, int64_t i, float r[4]);
template <>
__device__ __forceinline__ void load4<float>(const float* p, int64_t i, float r[4]) {
  const f32x4 v = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(p + i));
  r[0] = v[0]; r[1] = v[1]; r[2] = v[2]; r[3] = v[3];
}
template <>
__device__ __forceinline__ void load4<bf16>(const bf16* p, int64_t i, float r[4]) {
  const u32x2 v = __builtin_nontemporal_load(reinterpret_cast<const u32x2*>(p + i));
  r[0] = __uint_as_float(v[0] << 16); r[1] = __uint_as_float(v[0] & 0xffff0000u);
  r[2] = __uint_as_float(v[1] << 16); r[3] = __uint_as_float(v[1] & 0xffff0000u);
}
template <typename S>
__device__ __forceinline__ void store4(S* p, int64_t i, const float r[4]);
template <>
__device__ __forceinline__ void store4<float>(float* p, int64_t i, const float r[4]) {
  __builtin_nontemporal_store(f32x4{r[0], r[1], r[2], r[3]}, reinterpret_cast<f32x4*>(p + i));
}
template <>
__device__ __forceinline__ void store4<bf16>(bf16* p, int64_t i, const float r[4]) {
  bf16x4 v;
  v[0] = (bf16)r[0]; v[1] = (bf16)r[1]; v[2] = (bf16)r[2]; v[3] = (bf16)r[3];
  u32x2 u;
  __builtin_memcpy(&u, &v, 8);
  __builtin_nontemporal_store(u, reinterpret_cast<u32x2*>(p + i));
}

// Pass 1: block b sums g^2 over its contiguous range in double; partial[b].
template <typename G>
__global__ void __launch_bounds__(NORM_THREADS) sumsq_partial(const G* __restrict__ g, int64_t n,
                                                              double* __restrict__ partial) {
  __shared__ double sm[16];
  const int64_t per = ((n + gridDim.x - 1) / gridDim.x + 3) & ~int64_t(3);
  const int64_t lo = per * blockIdx.x;
  const int64_t hi = lo + per < n ? lo + per : n;
  double acc = 0.0;
  int64_t i = lo + 4 * threadIdx.x;
  const int64_t B4 = 4 * (int64_t)blockDim.x;
  for (; i + 3 * B4 + 3 < hi; i += 4 * B4) {  // four independent 16-byte loads in flight
    float r[4][4];
#pragma unroll
    for (int k = 0; k < 4; ++k) load4<G>(g, i + k * B4, r[k]);
#pragma unroll
    for (int k = 0; k < 4; ++k)
      acc += (double)r[k][0] * r[k][0] + (double)r[k][1] * r[k][1] + (double)r[k][2] * r[k][2] +
             (double)r[k][3] * r[k][3];
  }
  for (; i + 3 < hi; i += 4 * blockDim.x) {
    float r[4];
    load4<G>(g, i, r);
    acc += (double)r[0] * r[0] + (double)r[1] * r[1] + (double)r[2] * r[2] + (double)r[3] * r[3];
  }
  for (; i < hi; ++i) { float r = to_f32(g[i]); acc += (double)r * r; }  // ragged tail
  acc = block_sum<double>(acc, sm);
  if (threadIdx.x == 0) partial[blockIdx.x] = acc;
}

// Pass 2: one block sums the partials in a fixed order and derives the clip coefficient and the
// non-finite flag.  out[0] = ||g||, out[1] = clip scale c; flag[0] = 1 when ||g|| is not finite;
// skipped[0] counts non-finite norms.
__global__ void __launch_bounds__(1024) norm_finish(const double* __restrict__ partial, int np,
                                                   float clip, float* __restrict__ out,
                                                   int* __restrict__ flag,
                                                   unsigned long long* __restrict__ skipped) {
  __shared__ double sm[16];
  double acc = 0.0;
  for (int i = threadIdx.x; i < np; i += blockDim.x) acc += partial[i];
  acc = block_sum<double>(acc, sm);
  if (threadIdx.x == 0) {
    const double nrm = sqrt(acc);
    const bool bad = !isfinite(nrm);
    float c = 1.0f;
    if (clip > 0.0f && !bad) c = (float)fmin(1.0, (double)clip / (nrm + 1e-6));
    out[0] = (float)nrm;
    out[1] = c;
    if (flag) flag[0] = bad ? 1 : 0;
    if (bad && skipped) skipped[0] += 1ull;
  }
}

// One element of the fused pass: the optimizer rule OPT on the clipped gradient gg, then the
// standard or Error-Feedback step.  x, m, v are updated in place; u is the update, xc the value
// the compute copy receives (x, or the predicted point of UPD_ADAMW_PREDICT).
template <int OPT>
__device__ __forceinline__ void step_elem(float gg, float& x, float& m, float& v, float up, bool ef,
                                          const UpdateScalars& hs, float& u, float& xc) {
  if constexpr (OPT == UPD_LION) {
    const float c = hs.b1 * m + hs.omb1 * gg;
    const float sg = (c > 0.f) ? 1.f : (c < 0.f ? -1.f : 0.f);
    u = hs.lr * (sg + hs.wd * x);
    m = hs.b2 * m + hs.omb2 * gg;
  } else if constexpr (OPT == UPD_NADAM) {
    m = hs.b1 * m + hs.omb1 * gg;
    v = hs.b2 * v + hs.omb2 * (gg * gg);
    const float denom = sqrtf(v / hs.bc2) + hs.eps;
    u = (hs.cg * gg + hs.cm * m) / denom + hs.lr * hs.wd * x;
  } else {
    m = hs.b1 * m + hs.omb1 * gg;
    v = hs.b2 * v + hs.omb2 * (gg * gg);
    u = hs.lr * ((m / hs.bc1) / (sqrtf(v / hs.bc2) + hs.eps) + hs.wd * x);
  }
  x = ef ? x - hs.one_plus_lam * u + hs.lam * up : x - u;
  xc = x;
  if constexpr (OPT == UPD_ADAMW_PREDICT) {  // AdamW once more from the updated state, not kept
    const float m2 = hs.b1 * m + hs.omb1 * gg;
    const float v2 = hs.b2 * v + hs.omb2 * (gg * gg);
    xc = x - hs.lr * ((m2 / hs.bc1n) / (sqrtf(v2 / hs.bc2n) + hs.eps) + hs.wd * x);
  }
}

template <typename G, typename S, bool EF, int OPT>
__device__ __forceinline__ void update_group(int64_t n, int64_t i, float* __restrict__ x,
                                             const G* __restrict__ g, float* __restrict__ m,
                                             float* __restrict__ v, float* __restrict__ up,
                                             S* __restrict__ shadow, const UpdateScalars& hs, float c,
                                             bool skip) {
  constexpr bool USES_V = OPT != UPD_LION;
  if (i >= n) return;
  if (i + 3 < n) {
    float xr[4], xc[4];
    load4<float>(x, i, xr);
    if (!skip) {
      float gr[4], mr[4], vr[4] = {0.f, 0.f, 0.f, 0.f}, ur[4] = {0.f, 0.f, 0.f, 0.f};
      load4<G>(g, i, gr);
      load4<float>(m, i, mr);
      if (USES_V) load4<float>(v, i, vr);
      if (EF) load4<float>(up, i, ur);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        float u;
        step_elem<OPT>(gr[j] * c, xr[j], mr[j], vr[j], ur[j], EF && hs.ef, hs, u, xc[j]);
        ur[j] = u;
      }
      store4<float>(x, i, xr);
      store4<float>(m, i, mr);
      if (USES_V) store4<float>(v, i, vr);
      if (EF) store4<float>(up, i, ur);
    } else {
#pragma unroll
      for (int j = 0; j < 4; ++j) xc[j] = xr[j];
    }
    if (shadow) store4<S>(shadow, i, xc);
  } else {
    for (int64_t k = i; k < n; ++k) {  // ragged tail of a flat vector whose length is not 4k
      float xv = x[k], xcv = xv;
      if (!skip) {
        float mm = m[k], vv = USES_V ? v[k] : 0.f, u;
        step_elem<OPT>(to_f32(g[k]) * c, xv, mm, vv, EF ? up[k] : 0.f, EF && hs.ef, hs, u, xcv);
        m[k] = mm;
        if (USES_V) v[k] = vv;
        if (EF) up[k] = u;
        x[k] = xv;
      }
      if (shadow) shadow[k] = from_f32<S>(xcv);
    }
  }
}

// Each thread owns V groups of 4 consecutive elements, the groups one block-width apart so that
// every load instruction of a wave covers contiguous memory.
template <typename G, typename S, bool EF, int V, int OPT>
__global__ void __launch_bounds__(256) fused_update(int64_t n, float* __restrict__ x,
                                                    const G* __restrict__ g,
                                                    float* __restrict__ m, float* __restrict__ v,
                                                    float* __restrict__ up, S* __restrict__ shadow,
                                                    UpdateScalars hs, const float* __restrict__ clip,
                                                    const int* __restrict__ skip_flag) {
  const bool skip = hs.apply == 0 || (skip_flag && skip_flag[0] != 0);
  const float c = clip ? clip[0] : 1.0f;
  const int64_t i0 = 4 * ((int64_t)blockIdx.x * blockDim.x * V + threadIdx.x);
#pragma unroll
  for (int k = 0; k < V; ++k)
    update_group<G, S, EF, OPT>(n, i0 + 4 * (int64_t)k * blockDim.x, x, g, m, v, up, shadow, hs, c, skip);
}

// Resident variant: a grid of a few blocks per CU walks the vector (V groups per thread and
// pass), so that the pass shares the CUs with kernels of other streams instead of queueing a
// block per 1024 elements in front of them.
template <typename G, typename S, bool EF, int V, int OPT>
__global__ void __launch_bounds__(256) fused_update_resident(int64_t n, float* __restrict__ x,
                                                             const G* __restrict__ g,
                                                             float* __restrict__ m, float* __restrict__ v,
                                                             float* __restrict__ up, S* __restrict__ shadow,
                                                             UpdateScalars hs, const float* __restrict__ clip,
                                                             const int* __restrict__ skip_flag) {
  const bool skip = hs.apply == 0 || (skip_flag && skip_flag[0] != 0);
  const float c = clip ? clip[0] : 1.0f;
  const int64_t groups = (n + 3) / 4, stride = (int64_t)gridDim.x * blockDim.x * V;
  for (int64_t q = (int64_t)blockIdx.x * blockDim.x * V + threadIdx.x; q < groups; q += stride) {
#pragma unroll
    for (int k = 0; k < V; ++k)
      update_group<G, S, EF, OPT>(n, 4 * (q + (int64_t)k * blockDim.x), x, g, m, v, up, shadow, hs, c, skip);
  }
}

// Adan (Xie et al.) as the update function, one element group of 4: the clipped gradient gg, its
// difference from the clipped gradient of the previous update (0 at the first), the three averages
// m (gradient), d (differences), n (squared gg + b2 diff), then
//   u = lr ((m / bc1 + b2 d / bc2) / (sqrt(n / bc3) + eps) + wd x_t)
// and the standard or Error-Feedback step; g_last receives gg.  52 bytes per element with a bf16
// gradient and copy: x, m, n, d, g_last, u_prev read and written, g read, the copy written.
template <typename G, typename S, bool EF>
__device__ __forceinline__ void adan_group(int64_t n, int64_t i, float* __restrict__ x, const G* __restrict__ g,
                                           float* __restrict__ m, float* __restrict__ nn, float* __restrict__ d,
                                           float* __restrict__ gl, float* __restrict__ up, S* __restrict__ shadow,
                                           const UpdateScalars& hs, float c, bool skip) {
  if (i >= n) return;
  auto elem = [&](float gg, float& xv, float& mv, float& nv, float& dv, float& gv, float& uv) {
    const float diff = hs.first ? 0.f : gg - gv;
    mv = hs.b1 * mv + hs.omb1 * gg;
    dv = hs.b2 * dv + hs.omb2 * diff;
    const float q = gg + hs.b2 * diff;
    nv = hs.b3 * nv + hs.omb3 * (q * q);
    const float u = hs.lr * ((mv / hs.bc1 + hs.b2 * dv / hs.bc2) / (sqrtf(nv / hs.bc3) + hs.eps) + hs.wd * xv);
    xv = (EF && hs.ef) ? xv - hs.one_plus_lam * u + hs.lam * uv : xv - u;
    gv = gg;
    uv = u;
  };
  if (i + 3 < n) {
    float xr[4];
    load4<float>(x, i, xr);
    if (!skip) {
      float gr[4], mr[4], nr[4], dr[4], lr[4], ur[4] = {0.f, 0.f, 0.f, 0.f};
      load4<G>(g, i, gr);
      load4<float>(m, i, mr);
      load4<float>(nn, i, nr);
      load4<float>(d, i, dr);
      load4<float>(gl, i, lr);
      if (EF) load4<float>(up, i, ur);
#pragma unroll
      for (int j = 0; j < 4; ++j) elem(gr[j] * c, xr[j], mr[j], nr[j], dr[j], lr[j], ur[j]);
      store4<float>(x, i, xr);
      store4<float>(m, i, mr);
      store4<float>(nn, i, nr);
      store4<float>(d, i, dr);
      store4<float>(gl, i, lr);
      if (EF) store4<float>(up, i, ur);
    }
    if (shadow) store4<S>(shadow, i, xr);
  } else {
    for (int64_t k = i; k < n; ++k) {  // ragged tail
      float xv = x[k];
      if (!skip) {
        float mv = m[k], nv = nn[k], dv = d[k], gv = gl[k], uv = EF ? up[k] : 0.f;
        elem(to_f32(g[k]) * c, xv, mv, nv, dv, gv, uv);
        x[k] = xv; m[k] = mv; nn[k] = nv; d[k] = dv; gl[k] = gv;
        if (EF) up[k] = uv;
      }
      if (shadow) shadow[k] = from_f32<S>(xv);
    }
  }
}

// Grid-stride pass: a resident grid (blocks > 0 at launch) or one group of 4 elements per thread.
template <typename G, typename S, bool EF>
__global__ void __launch_bounds__(256) fused_update_adan(int64_t n, float* __restrict__ x, const G* __restrict__ g,
                                                         float* __restrict__ m, float* __restrict__ nn,
                                                         float* __restrict__ d, float* __restrict__ gl,
                                                         float* __restrict__ up, S* __restrict__ shadow,
                                                         UpdateScalars hs, const float* __restrict__ clip,
                                                         const int* __restrict__ skip_flag) {
  const bool skip = hs.apply == 0 || (skip_flag && skip_flag[0] != 0);
  const float c = clip ? clip[0] : 1.0f;
  const int64_t groups = (n + 3) / 4, stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; q < groups; q += stride)
    adan_group<G, S, EF>(n, 4 * q, x, g, m, nn, d, gl, up, shadow, hs, c, skip);
}

template <typename S>
__global__ void __launch_bounds__(256) cast_copy(int64_t n, const float* __restrict__ src,
                                                 S* __restrict__ dst) {
  const int64_t i = 4 * ((int64_t)blockIdx.x * blockDim.x + threadIdx.x);
  if (i + 3 < n) {
    float r[4];
    load4<float>(src, i, r);
    store4<S>(dst, i, r);
  } else {
    for (int64_t k = i; k < n; ++k) dst[k] = from_f32<S>(src[k]);
  }
}

// Streaming copy of n16 16-byte chunks, four per thread in flight (one block-width apart), with
// non-temporal loads and stores: the practical HBM ceiling the update pass is compared against.
__global__ void __launch_bounds__(256) stream_copy(int64_t n16, const u32x4* __restrict__ src,
                                                   u32x4* __restrict__ dst) {
  const int64_t i0 = (int64_t)blockIdx.x * blockDim.x * 4 + threadIdx.x;
  u32x4 r[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int64_t i = i0 + (int64_t)k * blockDim.x;
    if (i < n16) r[k] = __builtin_nontemporal_load(src + i);
  }
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int64_t i = i0 + (int64_t)k * blockDim.x;
    if (i < n16) __builtin_nontemporal_store(r[k], dst + i);
  }
}

__global__ void __launch_bounds__(256) zero_bytes(int64_t n16, int4* __restrict__ p) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n16) p[i] = make_int4(0, 0, 0, 0);
}

template <typename G, typename S, bool EF, int OPT>
void launch_update_o(int64_t n, float* x, const void* g, float* m, float* v, float* up,
                     void* shadow, const UpdateScalars& hs, const float* clip, const int* flag,
                     int blocks, hipStream_t st) {
  constexpr int V = 1;
  const int64_t groups = cdiv(n, 4);
  if (blocks > 0 && groups > (int64_t)blocks * 256 * 4) {
    fused_update_resident<G, S, EF, 4, OPT><<<blocks, 256, 0, st>>>(n, x, (const G*)g, m, v, up, (S*)shadow,
                                                                    hs, clip, flag);
    return;
  }
  const dim3 grid((unsigned)cdiv(groups, 256 * V));
  fused_update<G, S, EF, V, OPT><<<grid, 256, 0, st>>>(n, x, (const G*)g, m, v, up, (S*)shadow, hs, clip,
                                                       flag);
}

template <typename G, typename S, bool EF>
void launch_update_t(int64_t n, float* x, const void* g, float* m, float* v, float* up,
                     void* shadow, const UpdateScalars& hs, const float* clip, const int* flag,
                     int blocks, hipStream_t st) {
  switch (hs.opt) {
    case UPD_LION: launch_update_o<G, S, EF, UPD_LION>(n, x, g, m, v, up, shadow, hs, clip, flag, blocks, st); break;
    case UPD_NADAM: launch_update_o<G, S, EF, UPD_NADAM>(n, x, g, m, v, up, shadow, hs, clip, flag, blocks, st); break;
    case UPD_ADAMW_PREDICT:
      launch_update_o<G, S, EF, UPD_ADAMW_PREDICT>(n, x, g, m, v, up, shadow, hs, clip, flag, blocks, st);
      break;
    default: launch_update_o<G, S, EF, UPD_ADAMW>(n, x, g, m, v, up, shadow, hs, clip, flag, blocks, st);
  }
}

// Partial sums of the norm's first pass for callers that cannot allocate (grad_norm_flat_noalloc):
// one array per GPU, held until the process ends.  Host code never passes its name to a kernel: the
// name is a host-side stand-in, and the device address comes from hipGetSymbolAddress, per device.
static __device__ __align__(256) double scratch[NORM_BLOCKS];

}  // namespace

size_t norm_scratch_bytes() { return NORM_BLOCKS * sizeof(double); }

#include <mutex>
double* norm_static_scratch(int* err) {
  static std::mutex mu;
  static double* addr[64] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess || dev < 0 || dev >= 64) {
    *err = e != hipSuccess ? (int)e : (int)hipErrorInvalidDevice;
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));  // with device `dev` current
    if (e != hipSuccess || !p) {
      *err = e != hipSuccess ? (int)e : (int)hipErrorInvalidSymbol;
      return nullptr;
    }
    addr[dev] = (double*)p;
  }
  *err = 0;
  return addr[dev];
}

void launch_grad_norm(const void* g, bool g_bf16, int64_t n, float clip, double* partial,
                      float* out2, int* flag, unsigned long long* skipped, int blocks, hipStream_t st) {
  const int nb = blocks > 0 && blocks < NORM_BLOCKS ? blocks : NORM_BLOCKS;
  if (g_bf16)
    sumsq_partial<bf16><<<nb, NORM_THREADS, 0, st>>>((const bf16*)g, n, partial);
  else
    sumsq_partial<float><<<nb, NORM_THREADS, 0, st>>>((const float*)g, n, partial);
  norm_finish<<<1, 1024, 0, st>>>(partial, nb, clip, out2, flag, skipped);
}

void launch_fused_update(int64_t n, float* x, const void* g, bool g_bf16, float* m, float* v,
                         float* up, void* shadow, int shadow_kind, const UpdateScalars& hs,
                         const float* clip, const int* flag, int blocks, hipStream_t st) {
  // shadow_kind: 0 none, 1 fp32, 2 bf16.  EF instantiation whenever an EF buffer is present.
  const bool ef = up != nullptr;
#define UPD(G, S, E) launch_update_t<G, S, E>(n, x, g, m, v, up, shadow, hs, clip, flag, blocks, st)
  if (g_bf16) {
    if (shadow_kind == 2) { if (ef) UPD(bf16, bf16, true); else UPD(bf16, bf16, false); }
    else if (shadow_kind == 1) { if (ef) UPD(bf16, float, true); else UPD(bf16, float, false); }
    else { if (ef) UPD(bf16, float, true); else UPD(bf16, float, false); }
  } else {
    if (shadow_kind == 2) { if (ef) UPD(float, bf16, true); else UPD(float, bf16, false); }
    else if (shadow_kind == 1) { if (ef) UPD(float, float, true); else UPD(float, float, false); }
    else { if (ef) UPD(float, float, true); else UPD(float, float, false); }
  }
#undef UPD
}

void launch_fused_update_adan(int64_t n, float* x, const void* g, bool g_bf16, float* m, float* nn, float* d,
                              float* g_last, float* up, void* shadow, int shadow_kind, const UpdateScalars& hs,
                              const float* clip, const int* flag, int blocks, hipStream_t st) {
  const int64_t groups = cdiv(n, 4);
  const unsigned grid = (unsigned)(blocks > 0 && groups > (int64_t)blocks * 256 ? blocks : cdiv(groups, 256));
  const bool ef = up != nullptr;
#define ADAN(G, S, E) \
  fused_update_adan<G, S, E><<<grid, 256, 0, st>>>(n, x, (const G*)g, m, nn, d, g_last, up, (S*)shadow, hs, clip, flag)
  if (g_bf16) {
    if (shadow_kind == 2) { if (ef) ADAN(bf16, bf16, true); else ADAN(bf16, bf16, false); }
    else { if (ef) ADAN(bf16, float, true); else ADAN(bf16, float, false); }
  } else {
    if (shadow_kind == 2) { if (ef) ADAN(float, bf16, true); else ADAN(float, bf16, false); }
    else { if (ef) ADAN(float, float, true); else ADAN(float, float, false); }
  }
#undef ADAN
}

void launch_cast_copy(int64_t n, const float* src, void* dst, bool dst_bf16, hipStream_t st) {
  const dim3 grid((unsigned)cdiv(cdiv(n, 4), 256));
  if (dst_bf16) cast_copy<bf16><<<grid, 256, 0, st>>>(n, src, (bf16*)dst);
  else cast_copy<float><<<grid, 256, 0, st>>>(n, src, (float*)dst);
}

void launch_stream_copy(void* dst, const void* src, int64_t bytes, hipStream_t st) {
  const int64_t n16 = bytes / 16;
  if (n16 == 0) return;
  stream_copy<<<(unsigned)cdiv(n16, 256 * 4), 256, 0, st>>>(n16, (const u32x4*)src, (u32x4*)dst);
}

void launch_zero(void* p, int64_t bytes, hipStream_t st) {
  // bytes must be a multiple of 16 (every region the stage clears is 256-byte aligned)
  const int64_t n16 = bytes / 16;
  if (n16 == 0) return;
  zero_bytes<<<(unsigned)cdiv(n16, 256), 256, 0, st>>>(n16, (int4*)p);
}
