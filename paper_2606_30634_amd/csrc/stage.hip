// Host side of the stage library: arena layout, named tensors, the weight-version and
// gradient-buffer bookkeeping of the delayed update, and the kernel sequences of forward,
// backward and update.  Every device operation is a kernel of this library on the stage's stream.
//
// Bookkeeping (PipeDream-2BW, §2; Alg. 1): compute version v = step mod 2 holds x_step while the
// microbatches of that step run forward and backward; gradient buffer step mod (max_delay + 1)
// accumulates g_step; delayed_update(t) reads g_{t-tau} (delay tau, 1 in Alg. 1; App. C for a
// larger fixed delay) and writes x_{t+1} into version (t+1) mod 2, which no pending microbatch
// reads any more.  Error Feedback of iteration t uses EF buffer t mod tau, which holds the update
// formed tau iterations earlier and receives this one.
#include <cmath>
#include <cstdio>
#include <algorithm>
#include <cstring>
#include <string>
#include <vector>

#include "../../include/asyncstage.h"
#include "common.h"
#include "kernels.h"

namespace {

thread_local std::string g_err;

int fail(int code, const std::string& msg) {
  g_err = msg;
  return code;
}

#define HIP_OK(expr)                                                                   \
  do {                                                                                 \
    hipError_t e_ = (expr);                                                            \
    if (e_ != hipSuccess) return fail(STAGE_EHIP, std::string(#expr) + ": " + hipGetErrorString(e_)); \
  } while (0)

constexpr size_t ALIGN = 256;
size_t up(size_t x) { return (x + ALIGN - 1) / ALIGN * ALIGN; }

struct BlockOff {  // element offsets of one block's weights in the flat parameter vector
  int64_t attn_norm, wqkv, wo, ffn_norm, wgu, wdown;
};

struct BlockAct {
  void *x, *n1, *qkv, *o, *h, *n2, *gu, *z;
  float *rstd1, *lse, *rstd2;
  float* o32 = nullptr;  // bf16 stage: the attention output in fp32 (for the backward's delta)
};

struct Slot {
  std::vector<BlockAct> blk;
  void* y;          // output of the last block [T, d]
  void *hf;         // final norm output (last stage)
  float *rstdf, *logits, *lse_ce;  // head: final-norm statistics, fp32 logits, their row lse
  int32_t *tokens, *targets;
  // first stage: the microbatch's positions sorted by token (stable) and the start of each token's
  // run, sorted at forward time on the weight-gradient stream (the tokens are known then); the
  // backward's embedding-gradient scatter waits for ev_sort
  uint32_t *sorted_tok = nullptr, *sorted_pos = nullptr;
  int32_t* row_start = nullptr;
  hipEvent_t ev_sort = nullptr;
  int64_t step = -1;
  bool pending = false;
};

}  // namespace

struct stage {
  stage_shape_t sh;
  hipStream_t st;
  // The delayed update runs on its own stream: it reads the gradient of an earlier step and
  // writes the master state and the other weight version, none of which the forward / backward
  // of the current step touch, so the two overlap.  ev_bwd[p] marks the end of the last backward
  // of a step of parity p (its gradient and its use of weight version p); ev_upd the end of the
  // last update, which the stage stream waits for before anything enqueued after it.
  hipStream_t ust = nullptr;
  hipEvent_t ev_bwd[2] = {nullptr, nullptr}, ev_upd = nullptr, ev_now = nullptr;
  bool ev_bwd_set[2] = {false, false};
  // ev_grad[j]: the end of the last backward that wrote gradient buffer j (one per buffer of the
  // delay ring; with max_delay 1 the same points as ev_bwd)
  hipEvent_t ev_grad[STAGE_MAX_DELAY + 1] = {};
  bool ev_grad_set[STAGE_MAX_DELAY + 1] = {};
  // Overlap mode (stage_set_update_overlap): the stage stream does not wait for an update as a
  // whole; ev_upd_v[v] marks the end of the update that wrote compute version v, ev_upd_g[j] of the
  // one that read gradient buffer j, and the first stage-stream call that reads that version or
  // overwrites that buffer waits on it (the flags say a wait is still owed).
  int overlap = 0;  // 0 off, 1 on, 2 on with the update's elementwise pass deferred (pend)
  hipEvent_t ev_upd_v[2] = {}, ev_upd_g[STAGE_MAX_DELAY + 1] = {};
  bool upd_owed_v[2] = {}, upd_owed_g[STAGE_MAX_DELAY + 1] = {}, upd_owed_all = false;
  // Mode 2: the elementwise pass of the last delayed_update waits on the host as chunks
  // [offset, offset + count) of the flat vector.  Each stage_backward that reaches a block's
  // attention backward launches the next chunk on the update stream beside it (that work keeps the
  // matrix cores busy and leaves HBM bandwidth idle, where the forward's products beside a whole
  // pass would share it), and every call that needs the update's results launches the rest first.
  // The other fields are the pass's arguments.
  struct PendingPass {
    std::vector<std::pair<int64_t, int64_t>> chunks;
    size_t next = 0;
    const float* g = nullptr;
    float* up = nullptr;
    void* shadow = nullptr;
    UpdateScalars hs{};
    const float* clip = nullptr;
    const int* flag = nullptr;
    double bytes = 0;  // HBM bytes per element
    int vout = 0, gb = 0;
    bool apply = false;
  } pend;
  int last_mb = 1;  // microbatches per step of the last stage_backward (attention backwards per block)
  // The weight-gradient products (fp32 output) of a backward run on a second stream of their own,
  // beside the activation-gradient chain: ev_m2s orders one after the stage stream's work so far,
  // ev_wg[k] marks the end of the last product of kind k (the stage stream waits on it before it
  // overwrites a buffer that product reads), ev_wjoin joins the stream back at the end.
  // They go there only when the stage's products underfill the chip (wgrad_side): a block's
  // [tokens, d_model] activation-gradient product of fewer than two 256 x 256 tiles per compute
  // unit.  Products that fill it gain nothing from a second stream and would only run each other's
  // kernels slower (measured on the large workload: 367 ms per step either way), so they run in
  // order on the stage stream.
  hipStream_t wst = nullptr;
  bool wgrad_side = true;
  hipEvent_t ev_m2s = nullptr, ev_wjoin = nullptr, ev_wg[5] = {};
  bool bf;
  size_t esz;  // bytes per compute element
  int T, qkvw, hqd;
  // flat parameter layout
  int64_t n_flat = 0, off_embed = -1, off_final = -1, off_head = -1;  // off_head = off_embed when tied
  std::vector<BlockOff> boff;
  // flat vectors
  // ng = max_delay + 1 gradient buffers (step s accumulates into s mod ng) and max_delay EF
  // buffers (iteration t of a delay-tau run uses u_ring[t mod tau]; u_prev = u_ring[0])
  int ndelay = 1, ng = 2;
  float *master, *m, *v, *u_prev, *grad[STAGE_MAX_DELAY + 1], *u_ring[STAGE_MAX_DELAY];
  // Adan's extra state (shapes with optimizer 2): the average of gradient differences and the
  // clipped gradient of the previous update
  float *adan_d = nullptr, *adan_gl = nullptr;
  void* ver[2];
  // scratch
  void *dA, *dB, *dh, *dn, *dgu, *do_, *dqkv, *dlog, *dhf;
  float *delta, *rms_part, *row_loss, *cos_t, *sin_t, *norm_out, *upd_norm_out;
  double *norm_part, *upd_norm_part;
  float* gemm_ws;
  int* flag;
  unsigned long long* skipped;
  int32_t* sort_ws;  // the token sort's scratch (its sorts run in order on one stream)
  std::vector<Slot> slots;
  // bookkeeping
  int64_t version_step[2] = {-1, -1};
  int64_t grad_step[STAGE_MAX_DELAY + 1];
  int grad_count[STAGE_MAX_DELAY + 1];
  bool grad_consumed[STAGE_MAX_DELAY + 1];
  int64_t next_t = 0;
  int64_t n_updates = 0;
  unsigned long long skipped_seen = 0;
  // kernel-class timing
  struct ProfRec { int cls; hipEvent_t a, b; double work; };
  bool prof_on = false;
  std::vector<ProfRec> prof_pending;
  std::vector<hipEvent_t> prof_free;
  double prof_ms[STAGE_PROF_NCLASS] = {}, prof_work[STAGE_PROF_NCLASS] = {};
  int64_t prof_n[STAGE_PROF_NCLASS] = {};
  // Muon (shapes with optimizer 1): the blocks' weight matrices, grouped by their wide-orientation
  // shape for the batched Newton-Schulz products, and the ranges of the flat vector outside them
  // (AdamW: embedding, gains, padding)
  struct MuonGroup { int m, n, nb; bool carry; float* X[2]; bf16* S[2]; void* A; void* P; };
  std::vector<MuonMat> muon;
  std::vector<MuonGroup> mgroups;
  std::vector<std::pair<int64_t, int64_t>> adamw_ranges;  // (offset, count)
  MuonMat* muon_tab = nullptr;
  double* muon_part = nullptr;
  float* muon_norm = nullptr;
  int muon_nblk = 0, muon_ntile = 0;
  // named tensors
  struct Named { std::string name; void* ptr; int64_t numel; int32_t dtype; };
  std::vector<Named> named;

  void* wptr(int ver_idx, int64_t off) const { return (char*)ver[ver_idx] + off * esz; }
};

namespace {

hipEvent_t prof_event(stage* S) {
  if (!S->prof_free.empty()) {
    hipEvent_t e = S->prof_free.back();
    S->prof_free.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  (void)hipEventCreate(&e);
  return e;
}

void prof_collect(stage* S) {
  for (auto& r : S->prof_pending) {
    float ms = 0.f;
    (void)hipEventElapsedTime(&ms, r.a, r.b);
    S->prof_ms[r.cls] += ms;
    S->prof_work[r.cls] += r.work;
    S->prof_n[r.cls] += 1;
    S->prof_free.push_back(r.a);
    S->prof_free.push_back(r.b);
  }
  S->prof_pending.clear();
}

// Runs `launch` bracketed by an event pair on its stream (the stage stream unless `on` is given)
// when timing is enabled.
template <typename F>
void timed(stage* S, int cls, double work, F&& launch, hipStream_t on = nullptr) {
  if (!S->prof_on) { launch(); return; }
  if (!on) on = S->st;
  hipEvent_t a = prof_event(S), b = prof_event(S);
  (void)hipEventRecord(a, on);
  launch();
  (void)hipEventRecord(b, on);
  S->prof_pending.push_back({cls, a, b, work});
  if (S->prof_pending.size() > 4096) {  // bound the number of live events
    (void)hipEventSynchronize(b);
    prof_collect(S);
  }
}

// Overlap mode 2: launches the next deferred chunk of the update pass on the update stream and
// moves the update's completion events past it (a stage-stream wait issued before the launch would
// not cover the chunk, so every such wait is preceded by flush_pending).
void launch_pending_chunk(stage* S) {
  auto& p = S->pend;
  const int64_t o = p.chunks[p.next].first, n = p.chunks[p.next].second;
  ++p.next;
  timed(S, STAGE_PROF_UPDATE, p.bytes * n, [&] {
    launch_fused_update(n, S->master + o, p.g + o, false, S->m + o, S->v + o, p.up ? p.up + o : nullptr,
                        (char*)p.shadow + o * S->esz, S->bf ? 2 : 1, p.hs, p.clip, p.flag, device_cu_count(),
                        S->ust);
  }, S->ust);
  (void)hipEventRecord(S->ev_upd, S->ust);
  (void)hipEventRecord(S->ev_upd_v[p.vout], S->ust);
  if (p.apply) (void)hipEventRecord(S->ev_upd_g[p.gb], S->ust);
  if (p.next == p.chunks.size()) {
    p.chunks.clear();
    p.next = 0;
  }
}

void flush_pending(stage* S) {
  while (!S->pend.chunks.empty()) launch_pending_chunk(S);
}

// activation products on the stage stream (no split-K: the workspace belongs to the
// weight-gradient stream)
void run_gemm(stage* S, GemmArgs g) {
  g.ws = nullptr;
  g.ws_elems = 0;
  timed(S, STAGE_PROF_GEMM, 2.0 * g.M * g.N * g.K, [&] { launch_gemm(S->bf, g, S->st); });
}

enum { WG_DOWN = 0, WG_GU = 1, WG_O = 2, WG_QKV = 3, WG_HEAD = 4 };

// weight-gradient product of kind k on the weight-gradient stream, after everything enqueued on
// the stage stream so far (its inputs)
void run_wgrad(stage* S, GemmArgs g, int k) {
  if (!S->wgrad_side) {  // in order on the stage stream, with the split-K workspace
    g.ws = S->gemm_ws;
    g.ws_elems = S->gemm_ws ? GEMM_WS_ELEMS : 0;
    timed(S, STAGE_PROF_GEMM, 2.0 * g.M * g.N * g.K, [&] { launch_gemm(S->bf, g, S->st); });
    return;
  }
  (void)hipEventRecord(S->ev_m2s, S->st);
  (void)hipStreamWaitEvent(S->wst, S->ev_m2s, 0);
  g.ws = S->gemm_ws;
  g.ws_elems = S->gemm_ws ? GEMM_WS_ELEMS : 0;
  timed(S, STAGE_PROF_GEMM, 2.0 * g.M * g.N * g.K, [&] { launch_gemm(S->bf, g, S->wst); }, S->wst);
  (void)hipEventRecord(S->ev_wg[k], S->wst);
}

// the stage stream waits for the last weight-gradient product of kind k (and, the stream being in
// order, for every product issued before it)
void after_wgrad(stage* S, int k) {
  if (S->wgrad_side) (void)hipStreamWaitEvent(S->st, S->ev_wg[k], 0);
}

void join_wgrad(stage* S) {
  if (!S->wgrad_side) return;
  (void)hipEventRecord(S->ev_wjoin, S->wst);
  (void)hipStreamWaitEvent(S->st, S->ev_wjoin, 0);
}

double attn_fwd_flops(const stage* S) {  // QK^T and PV over the causal triangle
  const stage_shape_t& sh = S->sh;
  return 4.0 * sh.micro_batch * sh.n_heads * sh.head_dim * (double)sh.seq_len * (sh.seq_len + 1) / 2.0;
}

int validate(const stage_shape_t* s) {
  if (!s) return fail(STAGE_EINVAL, "null shape");
  if (s->n_blocks < 0 || s->d_model <= 0 || s->n_heads <= 0 || s->n_kv_heads <= 0 ||
      s->d_ffn <= 0 || s->seq_len <= 0 || s->micro_batch <= 0 || s->max_inflight <= 0)
    return fail(STAGE_EINVAL, "non-positive dimension");
  if (s->head_dim != 32 && s->head_dim != 64 && s->head_dim != 128)
    return fail(STAGE_EINVAL, "head_dim must be 32, 64 or 128");
  if (s->n_heads % s->n_kv_heads) return fail(STAGE_EINVAL, "n_heads % n_kv_heads != 0");
  if (s->d_model % 64 || s->d_ffn % 64) return fail(STAGE_EINVAL, "d_model, d_ffn must be multiples of 64");
  if (s->d_model > 4096) return fail(STAGE_EINVAL, "d_model > 4096 not supported");
  if (s->dtype != 0 && s->dtype != 1) return fail(STAGE_EINVAL, "dtype must be 0 (fp32) or 1 (bf16)");
  if (s->optimizer < 0 || s->optimizer > 2) return fail(STAGE_EINVAL, "optimizer must be 0, 1 (Muon workspace) or 2 (Adan state)");
  if (s->max_delay < 0 || s->max_delay > STAGE_MAX_DELAY)
    return fail(STAGE_EINVAL, "max_delay must be in [0, " + std::to_string(STAGE_MAX_DELAY) + "]");
  if (s->vocab < 0 || s->vocab >= (1 << 20)) return fail(STAGE_EINVAL, "vocab out of range [0, 2^20)");
  if (s->first_stage && s->vocab >= (1 << 17))
    return fail(STAGE_EINVAL, "a first stage's vocab must be below 2^17 (embedding-gradient sort keys)");
  if (s->vocab > 0 && !s->first_stage && !s->last_stage)
    return fail(STAGE_EINVAL, "vocab > 0 needs an embedding (first_stage) or a head (last_stage)");
  if (s->first_stage && s->vocab == 0) return fail(STAGE_EINVAL, "first_stage requires vocab > 0");
  if (s->last_stage && s->vocab == 0) return fail(STAGE_EINVAL, "last_stage requires vocab > 0");
  if (s->tie_embedding && !(s->first_stage && s->last_stage))
    return fail(STAGE_EINVAL, "tie_embedding needs a stage with both the embedding and the head");
  const int64_t T = (int64_t)s->seq_len * s->micro_batch;
  if (T > (1 << 24)) return fail(STAGE_EINVAL, "too many tokens per microbatch");
  return STAGE_OK;
}

// Lays the arena out; with base == nullptr only computes the size.
size_t layout(stage* S, char* base) {
  const stage_shape_t& sh = S->sh;
  const int64_t d = sh.d_model, f = sh.d_ffn, hd = sh.head_dim;
  const int64_t T = (int64_t)sh.seq_len * sh.micro_batch;
  const int64_t qkvw = (int64_t)(sh.n_heads + 2 * sh.n_kv_heads) * hd, hqd = (int64_t)sh.n_heads * hd;
  const size_t esz = sh.dtype == 1 ? 2 : 4;
  // flat parameter vector: groups aligned to 64 elements (256 bytes of fp32)
  int64_t n = 0;
  auto take = [&](int64_t cnt) { int64_t o = n; n += (cnt + 63) / 64 * 64; return o; };
  S->boff.clear();
  S->off_embed = sh.first_stage ? take((int64_t)sh.vocab * d) : -1;
  for (int i = 0; i < sh.n_blocks; ++i) {
    BlockOff b;
    b.attn_norm = take(d);
    b.wqkv = take(qkvw * d);
    b.wo = take(d * hqd);
    b.ffn_norm = take(d);
    b.wgu = take(2 * f * d);
    b.wdown = take(d * f);
    S->boff.push_back(b);
  }
  S->off_final = sh.last_stage ? take(d) : -1;
  S->off_head = !sh.last_stage ? -1 : sh.tie_embedding ? S->off_embed : take((int64_t)sh.vocab * d);
  S->n_flat = n;
  size_t off = 0;
  auto carve = [&](size_t bytes) -> void* { void* p = base ? base + off : nullptr; off += up(bytes); return p; };
  S->master = (float*)carve(n * 4);
  S->m = (float*)carve(n * 4);
  S->v = (float*)carve(n * 4);
  S->ndelay = sh.max_delay > 1 ? sh.max_delay : 1;
  S->ng = S->ndelay + 1;
  for (int j = 0; j < S->ndelay; ++j) S->u_ring[j] = (float*)carve(n * 4);
  S->u_prev = S->u_ring[0];
  for (int j = 0; j < S->ng; ++j) S->grad[j] = (float*)carve(n * 4);
  S->ver[0] = carve(n * esz);
  S->ver[1] = carve(n * esz);
  S->adan_d = sh.optimizer == 2 ? (float*)carve(n * 4) : nullptr;
  S->adan_gl = sh.optimizer == 2 ? (float*)carve(n * 4) : nullptr;
  // activation slots
  S->slots.assign(sh.max_inflight, Slot());
  for (auto& sl : S->slots) {
    sl.blk.resize(sh.n_blocks);
    for (auto& b : sl.blk) {
      b.x = carve(T * d * esz);
      b.rstd1 = (float*)carve(T * 4);
      b.n1 = carve(T * d * esz);
      b.qkv = carve(T * qkvw * esz);
      b.o = carve(T * hqd * esz);
      b.o32 = sh.dtype == 1 ? (float*)carve(T * hqd * 4) : nullptr;
      b.lse = (float*)carve((int64_t)sh.micro_batch * sh.n_heads * sh.seq_len * 4);
      b.h = carve(T * d * esz);
      b.rstd2 = (float*)carve(T * 4);
      b.n2 = carve(T * d * esz);
      b.gu = carve(T * 2 * f * esz);
      b.z = carve(T * f * esz);
    }
    sl.y = carve(T * d * esz);
    sl.tokens = sh.first_stage ? (int32_t*)carve(T * 4) : nullptr;
    sl.sorted_tok = sh.first_stage ? (uint32_t*)carve(T * 4) : nullptr;
    sl.sorted_pos = sh.first_stage ? (uint32_t*)carve(T * 4) : nullptr;
    sl.row_start = sh.first_stage ? (int32_t*)carve(((int64_t)sh.vocab + 1) * 4) : nullptr;
    sl.targets = sh.last_stage ? (int32_t*)carve(T * 4) : nullptr;
    sl.hf = sh.last_stage ? carve(T * d * esz) : nullptr;
    sl.rstdf = sh.last_stage ? (float*)carve(T * 4) : nullptr;
    sl.logits = sh.last_stage ? (float*)carve(T * (int64_t)sh.vocab * 4) : nullptr;
    sl.lse_ce = sh.last_stage ? (float*)carve(T * 4) : nullptr;
  }
  // scratch shared by all calls
  S->dA = carve(T * d * esz);
  S->dB = carve(T * d * esz);
  S->dh = carve(T * d * esz);
  S->dn = carve(T * d * esz);
  S->dgu = carve(T * 2 * f * esz);
  S->do_ = carve(T * hqd * esz);
  S->dqkv = carve(T * qkvw * esz);
  S->delta = (float*)carve((int64_t)sh.micro_batch * sh.n_heads * sh.seq_len * 4);
  S->rms_part = (float*)carve(rms_partial_rows(T) * d * 4);
  S->norm_part = (double*)carve(norm_scratch_bytes());
  S->upd_norm_part = (double*)carve(norm_scratch_bytes());
  S->upd_norm_out = (float*)carve(2 * 4);
  S->gemm_ws = sh.dtype == 1 ? (float*)carve(GEMM_WS_ELEMS * 4) : nullptr;
  S->norm_out = (float*)carve(2 * 4);
  S->flag = (int*)carve(4);
  S->skipped = (unsigned long long*)carve(8);
  S->cos_t = (float*)carve((int64_t)sh.seq_len * (hd / 2) * 4);
  S->sin_t = (float*)carve((int64_t)sh.seq_len * (hd / 2) * 4);
  S->sort_ws = sh.first_stage ? (int32_t*)carve(token_sort_ws_elems((int)T) * 4) : nullptr;
  S->dlog = sh.last_stage ? carve(T * (int64_t)sh.vocab * esz) : nullptr;
  S->dhf = sh.last_stage ? carve(T * d * esz) : nullptr;
  S->row_loss = sh.last_stage ? (float*)carve(T * 4) : nullptr;
  // Muon: every block's wq, wk, wv, wo, wgate, wup, wdown; a group per wide-orientation shape
  // (m = min(rows, cols) <= n) holds the matrices' fp32 Newton-Schulz iterates [m, n] (ping-pong
  // on the fp32 stage; on the bf16 stage one, plus the bf16 hi/lo operand form [m, 2n]: ping-pong
  // too when m and n are multiples of 128, as the iterate then stays in that form), and their Gram
  // products A = X X^T [m, m] and P = b A + c A A in the compute type ([m, 2m] with each column
  // twice when the hi/lo form is carried), each kind contiguous over the group for the batched GEMMs
  S->muon.clear();
  S->mgroups.clear();
  S->adamw_ranges.clear();
  S->muon_tab = nullptr;
  if (sh.optimizer == 1) {
    const int64_t dkv = (int64_t)sh.n_kv_heads * hd;
    struct Mx { int64_t off; int rows, cols; };
    std::vector<Mx> mx;
    for (const BlockOff& b : S->boff) {
      mx.push_back({b.wqkv, (int)hqd, (int)d});
      mx.push_back({b.wqkv + hqd * d, (int)dkv, (int)d});
      mx.push_back({b.wqkv + hqd * d + dkv * d, (int)dkv, (int)d});
      mx.push_back({b.wo, (int)d, (int)hqd});
      mx.push_back({b.wgu, (int)f, (int)d});
      mx.push_back({b.wgu + f * d, (int)f, (int)d});
      mx.push_back({b.wdown, (int)d, (int)f});
    }
    std::vector<int> gidx(mx.size()), slot(mx.size());
    for (size_t k = 0; k < mx.size(); ++k) {
      const int m = std::min(mx[k].rows, mx[k].cols), nn = std::max(mx[k].rows, mx[k].cols);
      size_t gi = 0;
      while (gi < S->mgroups.size() && (S->mgroups[gi].m != m || S->mgroups[gi].n != nn)) ++gi;
      if (gi == S->mgroups.size())
        S->mgroups.push_back({m, nn, 0, false, {nullptr, nullptr}, {nullptr, nullptr}, nullptr, nullptr});
      gidx[k] = (int)gi;
      slot[k] = S->mgroups[gi].nb++;
    }
    for (auto& gr : S->mgroups) {
      const size_t mn = (size_t)gr.nb * gr.m * gr.n, mm = (size_t)gr.nb * gr.m * gr.m;
      gr.carry = sh.dtype == 1 && gemm_batched_tiles(gr.m, gr.m, 3 * gr.n) && gemm_batched_tiles(gr.m, gr.m, gr.m) &&
                 gemm_batched_tiles(gr.m, gr.n, 2 * gr.m);
      gr.X[0] = (float*)carve(mn * 4);
      gr.X[1] = sh.dtype == 1 ? nullptr : (float*)carve(mn * 4);
      gr.S[0] = sh.dtype == 1 ? (bf16*)carve(mn * 2 * 2) : nullptr;
      gr.S[1] = gr.carry ? (bf16*)carve(mn * 2 * 2) : nullptr;
      gr.A = carve(mm * esz);
      gr.P = carve(mm * esz * (gr.carry ? 2 : 1));
    }
    int blk = 0, tile = 0;
    for (size_t k = 0; k < mx.size(); ++k) {
      const auto& gr = S->mgroups[gidx[k]];
      MuonMat mm{};
      mm.off = mx[k].off;
      mm.rows = mx[k].rows;
      mm.cols = mx[k].cols;
      mm.trans = mx[k].rows > mx[k].cols ? 1 : 0;
      mm.blk0 = blk;
      mm.tile0 = tile;
      mm.sqrt_max = (float)std::sqrt((double)std::max(mm.rows, mm.cols));
      for (int q = 0; q < 2; ++q)
        mm.x[q] = gr.X[q] ? gr.X[q] + (size_t)slot[k] * gr.m * gr.n : nullptr;
      blk += (int)muon_chunks((int64_t)mm.rows * mm.cols);
      tile += (int)muon_tiles(mm.rows, mm.cols);
      S->muon.push_back(mm);
    }
    S->muon_nblk = blk;
    S->muon_ntile = tile;
    S->muon_tab = (MuonMat*)carve(S->muon.size() * sizeof(MuonMat));
    S->muon_part = (double*)carve((size_t)blk * 8);
    S->muon_norm = (float*)carve(S->muon.size() * 4);
    // the flat vector outside the matrices (every matrix starts and ends on a 64-element boundary)
    std::vector<std::pair<int64_t, int64_t>> iv;
    for (const auto& mm : S->muon) iv.push_back({mm.off, mm.off + (int64_t)mm.rows * mm.cols});
    std::sort(iv.begin(), iv.end());
    int64_t at = 0;
    for (const auto& r : iv) {
      if (r.first > at) S->adamw_ranges.push_back({at, r.first - at});
      at = std::max(at, r.second);
    }
    if (n > at) S->adamw_ranges.push_back({at, n - at});
  }
  return off;
}

void register_tensors(stage* S) {
  const stage_shape_t& sh = S->sh;
  const int64_t d = sh.d_model, f = sh.d_ffn, hd = sh.head_dim;
  const int64_t T = (int64_t)sh.seq_len * sh.micro_batch;
  const int32_t cdt = S->bf ? STAGE_DT_BF16 : STAGE_DT_F32;
  struct P { std::string name; int64_t off, numel; };
  std::vector<P> ps;
  if (S->off_embed >= 0) ps.push_back({"embed", S->off_embed, (int64_t)sh.vocab * d});
  for (int i = 0; i < sh.n_blocks; ++i) {
    const BlockOff& b = S->boff[i];
    const std::string p = "blk" + std::to_string(i) + ".";
    const int64_t nq = (int64_t)sh.n_heads * hd * d, nk = (int64_t)sh.n_kv_heads * hd * d;
    ps.push_back({p + "attn_norm", b.attn_norm, d});
    ps.push_back({p + "wq", b.wqkv, nq});
    ps.push_back({p + "wk", b.wqkv + nq, nk});
    ps.push_back({p + "wv", b.wqkv + nq + nk, nk});
    ps.push_back({p + "wo", b.wo, d * sh.n_heads * hd});
    ps.push_back({p + "ffn_norm", b.ffn_norm, d});
    ps.push_back({p + "wgate", b.wgu, f * d});
    ps.push_back({p + "wup", b.wgu + f * d, f * d});
    ps.push_back({p + "wdown", b.wdown, d * f});
  }
  if (S->off_final >= 0) ps.push_back({"final_norm", S->off_final, d});
  if (S->off_head >= 0 && S->off_head != S->off_embed) ps.push_back({"head", S->off_head, (int64_t)sh.vocab * d});
  struct V { std::string pre; void* base; size_t es; int32_t dt; };
  std::vector<V> vs = {{"", S->master, 4, STAGE_DT_F32}, {"m.", S->m, 4, STAGE_DT_F32},
                       {"v.", S->v, 4, STAGE_DT_F32},    {"u_prev.", S->u_prev, 4, STAGE_DT_F32}};
  for (int j = 1; j < S->ndelay; ++j) vs.push_back({"u_prev" + std::to_string(j) + ".", S->u_ring[j], 4, STAGE_DT_F32});
  for (int j = 0; j < S->ng; ++j) vs.push_back({"grad" + std::to_string(j) + ".", S->grad[j], 4, STAGE_DT_F32});
  if (S->adan_d) {
    vs.push_back({"adan_d.", S->adan_d, 4, STAGE_DT_F32});
    vs.push_back({"adan_gprev.", S->adan_gl, 4, STAGE_DT_F32});
  }
  vs.push_back({"w0.", S->ver[0], S->esz, cdt});
  vs.push_back({"w1.", S->ver[1], S->esz, cdt});
  for (const auto& vv : vs)
    for (const auto& p : ps)
      S->named.push_back({vv.pre + p.name, (char*)vv.base + p.off * vv.es, p.numel, vv.dt});
  for (const auto& vv : vs) {  // "flat.master", "flat.m", ..., "flat.grad0", ..., "flat.w1"
    const std::string pre = vv.pre.empty() ? "master" : vv.pre.substr(0, vv.pre.size() - 1);
    S->named.push_back({"flat." + pre, vv.base, S->n_flat, vv.dt});
  }
  const int64_t lse_n = (int64_t)sh.micro_batch * sh.n_heads * sh.seq_len;
  for (size_t si = 0; si < S->slots.size(); ++si) {
    const Slot& sl = S->slots[si];
    const std::string a = "act" + std::to_string(si) + ".";
    for (int i = 0; i < sh.n_blocks; ++i) {
      const BlockAct& b = sl.blk[i];
      const std::string p = a + "blk" + std::to_string(i) + ".";
      S->named.push_back({p + "x", b.x, T * d, cdt});
      S->named.push_back({p + "rstd1", b.rstd1, T, STAGE_DT_F32});
      S->named.push_back({p + "n1", b.n1, T * d, cdt});
      S->named.push_back({p + "qkv", b.qkv, T * S->qkvw, cdt});
      S->named.push_back({p + "o", b.o, T * S->hqd, cdt});
      if (b.o32) S->named.push_back({p + "o32", b.o32, T * S->hqd, STAGE_DT_F32});
      S->named.push_back({p + "lse", b.lse, lse_n, STAGE_DT_F32});
      S->named.push_back({p + "h", b.h, T * d, cdt});
      S->named.push_back({p + "rstd2", b.rstd2, T, STAGE_DT_F32});
      S->named.push_back({p + "n2", b.n2, T * d, cdt});
      S->named.push_back({p + "gu", b.gu, T * 2 * f, cdt});
      S->named.push_back({p + "z", b.z, T * f, cdt});
    }
    S->named.push_back({a + "x0", sh.n_blocks > 0 ? sl.blk[0].x : sl.y, T * d, cdt});
    S->named.push_back({a + "y", sl.y, T * d, cdt});
    if (sl.logits) S->named.push_back({a + "logits", sl.logits, T * (int64_t)sh.vocab, STAGE_DT_F32});
  }
}

GemmArgs gemm(int M, int N, int K, const void* A, int lda, bool ak, const void* B, int ldb, bool bk,
              void* C, int ldc, bool out_f32 = false, float beta = 0.f, const void* resid = nullptr) {
  GemmArgs g;
  g.M = M; g.N = N; g.K = K;
  g.A = A; g.lda = lda; g.a_kmajor = ak;
  g.B = B; g.ldb = ldb; g.b_kmajor = bk;
  g.C = C; g.ldc = ldc; g.out_f32 = out_f32; g.beta = beta; g.resid = resid;
  return g;
}

AttnArgs attn_args(const stage* S, const BlockAct& b) {
  AttnArgs a;
  a.B = S->sh.micro_batch; a.S = S->sh.seq_len; a.Hq = S->sh.n_heads; a.Hkv = S->sh.n_kv_heads;
  a.hd = S->sh.head_dim; a.qkv = b.qkv; a.o = b.o; a.lse = b.lse;
  a.dout = nullptr; a.dqkv = nullptr; a.delta = nullptr;
  a.o32 = b.o32;
  return a;
}

void block_forward(stage* S, int vi, BlockAct& b, const BlockOff& w, void* y) {
  const stage_shape_t& sh = S->sh;
  const int T = S->T, d = sh.d_model, f = sh.d_ffn;
  const bool bf = S->bf;
  hipStream_t st = S->st;
  launch_rmsnorm_fwd(bf, b.x, S->wptr(vi, w.attn_norm), b.n1, b.rstd1, T, d, sh.rms_eps, st);
  // QKV projection with RoPE on the query and key heads in the GEMM epilogue
  GemmArgs gq = gemm(T, S->qkvw, d, b.n1, d, true, S->wptr(vi, w.wqkv), d, true, b.qkv, S->qkvw);
  gq.epi = 2;
  gq.rope_cos = S->cos_t;
  gq.rope_sin = S->sin_t;
  gq.rope_cols = (sh.n_heads + sh.n_kv_heads) * sh.head_dim;
  gq.rope_hd = sh.head_dim;
  gq.rope_S = sh.seq_len;
  run_gemm(S, gq);
  timed(S, STAGE_PROF_ATTN_FWD, attn_fwd_flops(S), [&] { launch_attention_fwd(bf, attn_args(S, b), st); });
  run_gemm(S, gemm(T, d, S->hqd, b.o, S->hqd, true, S->wptr(vi, w.wo), S->hqd, true, b.h, d,
                       false, 0.f, b.x));
  launch_rmsnorm_fwd(bf, b.h, S->wptr(vi, w.ffn_norm), b.n2, b.rstd2, T, d, sh.rms_eps, st);
  // gate/up projection with the SwiGLU z = silu(gate) up in its epilogue
  GemmArgs gg = gemm(T, 2 * f, d, b.n2, d, true, S->wptr(vi, w.wgu), d, true, b.gu, 2 * f);
  gg.epi = 3;
  gg.glu = f;
  gg.out2 = b.z;
  gg.ld_out2 = f;
  run_gemm(S, gg);
  run_gemm(S, gemm(T, d, f, b.z, f, true, S->wptr(vi, w.wdown), f, true, y, d, false, 0.f, b.h));
}

// dy: gradient of the block output; writes the gradient of the block input into dx.
void block_backward(stage* S, int vi, BlockAct& b, const BlockOff& w, const void* dy, void* dx,
                    float* g, bool first) {
  const stage_shape_t& sh = S->sh;
  const int T = S->T, d = sh.d_model, f = sh.d_ffn;
  const bool bf = S->bf;
  const float beta = first ? 0.f : 1.f;
  hipStream_t st = S->st;
  // The weight gradients dW (+)= dY^T X run on the weight-gradient stream; before this stream
  // overwrites dgu, dh, dqkv or the previous block's dy, it waits for the product that read it.
  // down projection: dz = dy Wd with the SwiGLU backward in its epilogue (-> dgate | dup);
  // dWd (+)= dy^T z
  GemmArgs gz = gemm(T, f, d, dy, d, true, S->wptr(vi, w.wdown), f, false, S->dgu, 2 * f);
  gz.epi = 1;
  gz.aux = b.gu;
  gz.ld_aux = 2 * f;
  after_wgrad(S, WG_GU);
  run_gemm(S, gz);
  run_wgrad(S, gemm(d, f, T, dy, d, false, b.z, f, false, g + w.wdown, f, true, beta), WG_DOWN);
  // gate/up: dn2 = dgu Wgu ; dWgu (+)= dgu^T n2
  run_gemm(S, gemm(T, d, 2 * f, S->dgu, 2 * f, true, S->wptr(vi, w.wgu), d, false, S->dn, d));
  run_wgrad(S, gemm(2 * f, d, T, S->dgu, 2 * f, false, b.n2, d, false, g + w.wgu, d, true, beta), WG_GU);
  after_wgrad(S, WG_O);
  int np = launch_rmsnorm_bwd(bf, S->dn, b.h, b.rstd2, S->wptr(vi, w.ffn_norm), dy, S->dh, S->rms_part, T, d, st);
  launch_colsum_partials(S->rms_part, np, d, g + w.ffn_norm, !first, st);
  // output projection: do = dh Wo ; dWo (+)= dh^T o.  The attention backward's delta = rowsum(do o)
  // in the product's epilogue, from o in fp32 (the bf16 stage's forward keeps an fp32 copy whose P V
  // product took P as a hi / lo pair: delta then matches the P and dP the backward recomputes, where
  // o rounded to bf16 would leave every dS row a nonzero sum once attention sharpens)
  GemmArgs go = gemm(T, S->hqd, d, S->dh, d, true, S->wptr(vi, w.wo), S->hqd, false, S->do_, S->hqd);
  go.epi = 4;
  go.aux = bf ? (const void*)b.o32 : b.o;
  go.ld_aux = S->hqd;
  go.delta = S->delta;
  go.delta_hd = sh.head_dim;
  go.delta_S = sh.seq_len;
  run_gemm(S, go);
  run_wgrad(S, gemm(d, S->hqd, T, S->dh, d, false, b.o, S->hqd, false, g + w.wo, S->hqd, true, beta), WG_O);
  AttnArgs a = attn_args(S, b);
  a.dout = S->do_; a.dqkv = S->dqkv; a.delta = S->delta;
  a.delta_ready = true;  // computed with do above
  a.rope_cos = S->cos_t;  // dq, dk come back w.r.t. the unrotated projections
  a.rope_sin = S->sin_t;
  after_wgrad(S, WG_QKV);
  if (!S->pend.chunks.empty()) {
    // a deferred chunk of the update pass (overlap mode 2) starts with the attention backward
    (void)hipEventRecord(S->ev_now, st);
    (void)hipStreamWaitEvent(S->ust, S->ev_now, 0);
    launch_pending_chunk(S);
  }
  timed(S, STAGE_PROF_ATTN_BWD, 2.0 * attn_fwd_flops(S), [&] { launch_attention_bwd(bf, a, st); });
  // qkv projection: dn1 = dqkv Wqkv ; dWqkv (+)= dqkv^T n1
  run_gemm(S, gemm(T, d, S->qkvw, S->dqkv, S->qkvw, true, S->wptr(vi, w.wqkv), d, false, S->dn, d));
  run_wgrad(S, gemm(S->qkvw, d, T, S->dqkv, S->qkvw, false, b.n1, d, false, g + w.wqkv, d, true, beta), WG_QKV);
  after_wgrad(S, WG_DOWN);  // dx is the buffer the next-higher block's down-projection product read
  np = launch_rmsnorm_bwd(bf, S->dn, b.x, b.rstd1, S->wptr(vi, w.attn_norm), S->dh, dx, S->rms_part, T, d, st);
  launch_colsum_partials(S->rms_part, np, d, g + w.attn_norm, !first, st);
}

}  // namespace

extern "C" {

const char* stage_last_error(void) { return g_err.c_str(); }

size_t stage_required_bytes(const stage_shape_t* shape) {
  if (validate(shape) != STAGE_OK) return 0;
  stage tmp;
  tmp.sh = *shape;
  return layout(&tmp, nullptr);
}

int stage_init(const stage_shape_t* shape, void* arena, size_t arena_bytes, void* hip_stream,
               stage_t** out) {
  if (!out) return fail(STAGE_EINVAL, "null out");
  *out = nullptr;
  int rc = validate(shape);
  if (rc) return rc;
  if (!arena || ((uintptr_t)arena % ALIGN)) return fail(STAGE_EINVAL, "arena must be 256-byte aligned");
  stage* S = new stage();
  S->sh = *shape;
  for (int j = 0; j <= STAGE_MAX_DELAY; ++j) {
    S->grad_step[j] = -1;
    S->grad_count[j] = 0;
    S->grad_consumed[j] = true;
  }
  S->st = (hipStream_t)hip_stream;
  S->bf = shape->dtype == 1;
  S->esz = S->bf ? 2 : 4;
  S->T = shape->seq_len * shape->micro_batch;
  S->qkvw = (shape->n_heads + 2 * shape->n_kv_heads) * shape->head_dim;
  S->hqd = shape->n_heads * shape->head_dim;
  S->wgrad_side = (int64_t)(S->T / 256) * (shape->d_model / 256) < 2 * (int64_t)device_cu_count();
  const size_t need = layout(S, nullptr);
  if (arena_bytes < need) {
    delete S;
    return fail(STAGE_ENOSPACE, "arena holds " + std::to_string(arena_bytes) + " bytes, needs " + std::to_string(need));
  }
  layout(S, (char*)arena);
  register_tensors(S);
  {
    hipError_t e = hipStreamCreateWithFlags(&S->ust, hipStreamNonBlocking);
    if (e == hipSuccess) e = hipStreamCreateWithFlags(&S->wst, hipStreamNonBlocking);
    for (int k = 0; k < 5 && e == hipSuccess; ++k) e = hipEventCreateWithFlags(&S->ev_wg[k], hipEventDisableTiming);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&S->ev_m2s, hipEventDisableTiming);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&S->ev_wjoin, hipEventDisableTiming);
    for (int k = 0; k < 2 && e == hipSuccess; ++k) e = hipEventCreateWithFlags(&S->ev_bwd[k], hipEventDisableTiming);
    for (int k = 0; k < S->ng && e == hipSuccess; ++k)
      e = hipEventCreateWithFlags(&S->ev_grad[k], hipEventDisableTiming);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&S->ev_upd, hipEventDisableTiming);
    for (int k = 0; k < 2 && e == hipSuccess; ++k) e = hipEventCreateWithFlags(&S->ev_upd_v[k], hipEventDisableTiming);
    for (int k = 0; k < S->ng && e == hipSuccess; ++k)
      e = hipEventCreateWithFlags(&S->ev_upd_g[k], hipEventDisableTiming);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&S->ev_now, hipEventDisableTiming);
    for (auto& sl : S->slots)
      if (e == hipSuccess && shape->first_stage) e = hipEventCreateWithFlags(&sl.ev_sort, hipEventDisableTiming);
    if (e != hipSuccess) {
      stage_destroy(S);
      return fail(STAGE_EHIP, std::string("stage_init: ") + hipGetErrorString(e));
    }
  }
  launch_zero(arena, (int64_t)need, S->st);
  // RoPE tables: angle(p, i) = p * theta^(-2i/hd), evaluated in double
  const int half = shape->head_dim / 2;
  std::vector<float> c((size_t)shape->seq_len * half), s(c.size());
  for (int p = 0; p < shape->seq_len; ++p)
    for (int i = 0; i < half; ++i) {
      const double ang = p * std::pow((double)shape->rope_theta, -2.0 * i / shape->head_dim);
      c[(size_t)p * half + i] = (float)std::cos(ang);
      s[(size_t)p * half + i] = (float)std::sin(ang);
    }
  hipError_t e = hipMemcpyAsync(S->cos_t, c.data(), c.size() * 4, hipMemcpyHostToDevice, S->st);
  if (e == hipSuccess) e = hipMemcpyAsync(S->sin_t, s.data(), s.size() * 4, hipMemcpyHostToDevice, S->st);
  if (e == hipSuccess && S->muon_tab)
    e = hipMemcpyAsync(S->muon_tab, S->muon.data(), S->muon.size() * sizeof(MuonMat), hipMemcpyHostToDevice, S->st);
  if (e == hipSuccess) e = hipStreamSynchronize(S->st);
  if (e == hipSuccess) e = hipGetLastError();
  if (e != hipSuccess) {
    stage_destroy(S);
    return fail(STAGE_EHIP, std::string("stage_init: ") + hipGetErrorString(e));
  }
  *out = S;
  return STAGE_OK;
}

int stage_num_tensors(const stage_t* s, int32_t* count) {
  if (!s || !count) return fail(STAGE_EINVAL, "null argument");
  *count = (int32_t)s->named.size();
  return STAGE_OK;
}

int stage_tensor(const stage_t* s, int32_t idx, const char** name, void** dev_ptr, int64_t* numel,
                 int32_t* dtype) {
  if (!s || idx < 0 || idx >= (int32_t)s->named.size()) return fail(STAGE_EINVAL, "bad tensor index");
  const auto& t = s->named[idx];
  if (name) *name = t.name.c_str();
  if (dev_ptr) *dev_ptr = t.ptr;
  if (numel) *numel = t.numel;
  if (dtype) *dtype = t.dtype;
  return STAGE_OK;
}

int stage_tensor_by_name(const stage_t* s, const char* name, void** dev_ptr, int64_t* numel,
                         int32_t* dtype) {
  if (!s || !name) return fail(STAGE_EINVAL, "null argument");
  for (const auto& t : s->named)
    if (t.name == name) {
      if (dev_ptr) *dev_ptr = t.ptr;
      if (numel) *numel = t.numel;
      if (dtype) *dtype = t.dtype;
      return STAGE_OK;
    }
  return fail(STAGE_EINVAL, std::string("no tensor named ") + name);
}

int stage_join_update(stage_t* s) {
  if (!s) return fail(STAGE_EINVAL, "null stage");
  flush_pending(s);
  if (s->upd_owed_all) {
    HIP_OK(hipStreamWaitEvent(s->st, s->ev_upd, 0));
    s->upd_owed_all = false;
    for (int v = 0; v < 2; ++v) s->upd_owed_v[v] = false;
    for (int j = 0; j < s->ng; ++j) s->upd_owed_g[j] = false;
  }
  return STAGE_OK;
}

int stage_set_update_overlap(stage_t* s, int32_t on) {
  if (!s) return fail(STAGE_EINVAL, "null stage");
  if (on < 0 || on > 2) return fail(STAGE_EINVAL, "overlap mode must be 0, 1 or 2");
  if (on < 2) flush_pending(s);
  if (!on) stage_join_update(s);
  s->overlap = on;
  return STAGE_OK;
}

int stage_sync_weights(stage_t* s) {
  if (!s) return fail(STAGE_EINVAL, "null stage");
  stage_join_update(s);
  for (int k = 0; k < 2; ++k) launch_cast_copy(s->n_flat, s->master, s->ver[k], s->bf, s->st);
  HIP_OK(hipGetLastError());
  // the caller may have written the optimizer state: the next update waits for the whole stream
  s->ev_bwd_set[0] = s->ev_bwd_set[1] = false;
  for (int j = 0; j < s->ng; ++j) s->ev_grad_set[j] = false;
  s->version_step[s->next_t % 2] = s->next_t;
  s->version_step[(s->next_t + 1) % 2] = -1;
  return STAGE_OK;
}

int stage_forward(stage_t* s, int32_t slot, int64_t step, const int32_t* tokens, const void* x_in,
                  const int32_t* targets, void* y_out, float* loss_dev) {
  if (!s) return fail(STAGE_EINVAL, "null stage");
  const stage_shape_t& sh = s->sh;
  if (slot < 0 || slot >= sh.max_inflight) return fail(STAGE_EINVAL, "slot out of range");
  if (step < 0 || s->version_step[step % 2] != step)
    return fail(STAGE_ESTATE, "weights of step " + std::to_string(step) + " are not resident");
  if (sh.first_stage && !tokens) return fail(STAGE_EINVAL, "first stage needs tokens");
  if (!sh.first_stage && !x_in) return fail(STAGE_EINVAL, "non-first stage needs x_in");
  if (sh.last_stage && (!targets || !loss_dev)) return fail(STAGE_EINVAL, "last stage needs targets and loss_dev");
  Slot& sl = s->slots[slot];
  if (sl.pending) return fail(STAGE_ESTATE, "slot holds a microbatch whose backward is pending");
  const int vi = (int)(step % 2);
  if (vi == s->pend.vout) flush_pending(s);  // the deferred pass writes this version
  if (s->upd_owed_v[vi]) {
    HIP_OK(hipStreamWaitEvent(s->st, s->ev_upd_v[vi], 0));
    s->upd_owed_v[vi] = false;
  }
  const int T = s->T, d = sh.d_model;
  hipStream_t st = s->st;
  void* x0 = sh.n_blocks > 0 ? sl.blk[0].x : sl.y;
  if (sh.first_stage) {
    HIP_OK(hipMemcpyAsync(sl.tokens, tokens, (size_t)T * 4, hipMemcpyDeviceToDevice, st));
    launch_embed_gather(s->bf, sl.tokens, s->wptr(vi, s->off_embed), x0, T, d, sh.vocab, st);
    // the embedding gradient's sort needs only the tokens: beside the forward, where there is a
    // second stream
    hipStream_t ss = s->wgrad_side ? s->wst : st;
    if (ss != st) {
      HIP_OK(hipEventRecord(s->ev_m2s, st));
      HIP_OK(hipStreamWaitEvent(ss, s->ev_m2s, 0));
    }
    launch_token_sort(sl.tokens, T, sh.vocab, s->sort_ws, sl.sorted_tok, sl.sorted_pos, ss);
    launch_token_runs(sl.sorted_tok, T, sh.vocab, sl.row_start, nullptr, nullptr, nullptr, ss);
    HIP_OK(hipEventRecord(sl.ev_sort, ss));
  } else {
    HIP_OK(hipMemcpyAsync(x0, x_in, (size_t)T * d * s->esz, hipMemcpyDeviceToDevice, st));
  }
  for (int i = 0; i < sh.n_blocks; ++i) {
    void* y = i + 1 < sh.n_blocks ? sl.blk[i + 1].x : sl.y;
    block_forward(s, vi, sl.blk[i], s->boff[i], y);
  }
  if (sh.last_stage) {
    HIP_OK(hipMemcpyAsync(sl.targets, targets, (size_t)T * 4, hipMemcpyDeviceToDevice, st));
    launch_rmsnorm_fwd(s->bf, sl.y, s->wptr(vi, s->off_final), sl.hf, sl.rstdf, T, d, sh.rms_eps, st);
    run_gemm(s, gemm(T, sh.vocab, d, sl.hf, d, true, s->wptr(vi, s->off_head), d, true,
                            sl.logits, sh.vocab, true, 0.f));
    launch_ce_fwd(sl.logits, sl.targets, T, sh.vocab, sl.lse_ce, s->row_loss, st);
    launch_mean(s->row_loss, T, loss_dev, st);
  }
  if (y_out && !sh.last_stage)
    HIP_OK(hipMemcpyAsync(y_out, sl.y, (size_t)T * d * s->esz, hipMemcpyDeviceToDevice, st));
  HIP_OK(hipGetLastError());
  sl.step = step;
  sl.pending = true;
  return STAGE_OK;
}

int stage_backward(stage_t* s, int32_t slot, const void* dy, void* dx_out, int32_t microbatches_per_step) {
  if (!s) return fail(STAGE_EINVAL, "null stage");
  const stage_shape_t& sh = s->sh;
  if (slot < 0 || slot >= sh.max_inflight) return fail(STAGE_EINVAL, "slot out of range");
  Slot& sl = s->slots[slot];
  if (!sl.pending) return fail(STAGE_ESTATE, "slot holds no pending forward");
  if (!sh.last_stage && !dy) return fail(STAGE_EINVAL, "non-last stage needs dy");
  if (microbatches_per_step <= 0) return fail(STAGE_EINVAL, "microbatches_per_step must be positive");
  const int64_t step = sl.step;
  const int gb = (int)(step % s->ng), vi = (int)(step % 2);
  s->last_mb = microbatches_per_step;
  if (s->pend.apply && gb == s->pend.gb) flush_pending(s);  // the deferred pass reads this buffer
  if (s->upd_owed_g[gb]) {
    HIP_OK(hipStreamWaitEvent(s->st, s->ev_upd_g[gb], 0));
    s->upd_owed_g[gb] = false;
  }
  if (s->grad_step[gb] != step) {
    if (s->grad_step[gb] >= 0 && !s->grad_consumed[gb])
      return fail(STAGE_ESTATE, "gradient buffer still holds the unconsumed gradient of step " +
                                    std::to_string(s->grad_step[gb]));
    s->grad_step[gb] = step;
    s->grad_count[gb] = 0;
    s->grad_consumed[gb] = false;
  }
  const bool first = s->grad_count[gb] == 0;
  float* g = s->grad[gb];
  const int T = s->T, d = sh.d_model;
  const bool bf = s->bf;
  hipStream_t st = s->st;
  const void* cur = dy;
  bool head_wrote_embed = false;
  if (sh.last_stage) {
    launch_ce_bwd(bf, sl.logits, sl.targets, sl.lse_ce, T, sh.vocab, 1.0f / ((float)T * microbatches_per_step),
                  s->dlog, st);
    // dhf = dlogits W ; dW (+)= dlogits^T hf   (W the head matrix, or the tied embedding)
    run_gemm(s, gemm(T, d, sh.vocab, s->dlog, sh.vocab, true, s->wptr(vi, s->off_head), d, false,
                         s->dhf, d));
    run_wgrad(s, gemm(sh.vocab, d, T, s->dlog, sh.vocab, false, sl.hf, d, false, g + s->off_head, d,
                          true, first ? 0.f : 1.f), WG_HEAD);
    head_wrote_embed = s->off_head == s->off_embed;
    const int np = launch_rmsnorm_bwd(bf, s->dhf, sl.y, sl.rstdf, s->wptr(vi, s->off_final), nullptr, s->dA,
                                       s->rms_part, T, d, st);
    launch_colsum_partials(s->rms_part, np, d, g + s->off_final, !first, st);
    cur = s->dA;
  }
  for (int i = sh.n_blocks - 1; i >= 0; --i) {
    void* out = (cur == s->dA) ? s->dB : s->dA;
    block_backward(s, vi, sl.blk[i], s->boff[i], cur, out, g, first);
    cur = out;
  }
  if (sh.first_stage) {
    // the scatter reads the sorted positions and the activation gradient and writes the
    // embedding's rows, which only a tied head's weight-gradient product also writes: it runs
    // beside the remaining weight-gradient products
    const void* dx0 = cur;
    HIP_OK(hipStreamWaitEvent(st, sl.ev_sort, 0));
    if (head_wrote_embed) after_wgrad(s, WG_HEAD);
    launch_embed_scatter(bf, dx0, sl.sorted_pos, sl.row_start, sh.vocab, d, g + s->off_embed,
                         head_wrote_embed || !first, st);
  } else if (dx_out) {
    HIP_OK(hipMemcpyAsync(dx_out, cur, (size_t)T * d * s->esz, hipMemcpyDeviceToDevice, st));
  }
  join_wgrad(s);  // every weight gradient is in g
  HIP_OK(hipEventRecord(s->ev_bwd[vi], st));
  s->ev_bwd_set[vi] = true;
  HIP_OK(hipEventRecord(s->ev_grad[gb], st));
  s->ev_grad_set[gb] = true;
  HIP_OK(hipGetLastError());
  s->grad_count[gb] += 1;
  sl.pending = false;
  return STAGE_OK;
}

}  // extern "C"

namespace {

// Scalars of the fused elementwise pass for the k-th applied update (k >= 1 when apply): the
// AdamW bias corrections, Lion's betas, NAdam's momentum-schedule coefficients (mu_j = b1 (1 -
// 0.5 0.96^(j psi)), P_k = mu_1 ... mu_k, in double), and the bias corrections of update k + 1 for
// the weight prediction with the updated state.
UpdateScalars update_scalars(const update_hparams_t* hp, int64_t k, bool apply, bool ef) {
  UpdateScalars hs{};
  const double kk = apply ? (double)k : 0.0;
  hs.lr = hp->lr; hs.b1 = hp->beta1; hs.b2 = hp->beta2;
  hs.omb1 = 1.0f - hp->beta1; hs.omb2 = 1.0f - hp->beta2;
  hs.bc1 = apply ? (float)(1.0 - std::pow((double)hp->beta1, kk)) : 1.f;
  hs.bc2 = apply ? (float)(1.0 - std::pow((double)hp->beta2, kk)) : 1.f;
  hs.eps = hp->eps; hs.wd = hp->weight_decay; hs.lam = hp->ef_lambda;
  hs.one_plus_lam = 1.0f + hp->ef_lambda;
  hs.ef = ef ? 1 : 0;
  hs.apply = apply ? 1 : 0;
  hs.opt = hp->optimizer == 2 ? UPD_LION : hp->optimizer == 3 ? UPD_NADAM : hp->optimizer == 4 ? UPD_ADAN
           : hp->predict ? UPD_ADAMW_PREDICT : UPD_ADAMW;
  if (hs.opt == UPD_ADAN) {
    hs.b3 = hp->beta3;
    hs.omb3 = 1.0f - hp->beta3;
    hs.bc3 = apply ? (float)(1.0 - std::pow((double)hp->beta3, kk)) : 1.f;
    hs.first = k == 1 ? 1 : 0;
  }
  if (apply && hs.opt == UPD_NADAM) {
    auto mu = [&](int64_t j) { return (double)hp->beta1 * (1.0 - 0.5 * std::pow(0.96, (double)j * hp->nadam_psi)); };
    double prod = 1.0;
    for (int64_t j = 1; j <= k; ++j) prod *= mu(j);
    const double mk = mu(k), mn = mu(k + 1);
    hs.cg = (float)(hp->lr * (1.0 - mk) / (1.0 - prod));
    hs.cm = (float)(hp->lr * mn / (1.0 - prod * mn));
  }
  if (apply && hs.opt == UPD_ADAMW_PREDICT) {
    hs.bc1n = (float)(1.0 - std::pow((double)hp->beta1, kk + 1.0));
    hs.bc2n = (float)(1.0 - std::pow((double)hp->beta2, kk + 1.0));
  }
  return hs;
}

// Hyper-parameter checks shared by the stage and the flat update.
int check_update_hparams(const update_hparams_t* hp) {
  if (hp->optimizer < 0 || hp->optimizer > 4)
    return fail(STAGE_EINVAL, "optimizer must be 0 (AdamW), 1 (Muon), 2 (Lion), 3 (NAdam) or 4 (Adan)");
  if (hp->predict != 0 && hp->predict != 1) return fail(STAGE_EINVAL, "predict must be 0 or 1");
  if (hp->predict && (hp->optimizer != 0 || hp->ef_lambda != 0.f || hp->delay != 1))
    return fail(STAGE_EINVAL, "weight prediction (predict 1) needs AdamW, delay 1 and ef_lambda 0");
  return STAGE_OK;
}

}  // namespace

extern "C" {

int delayed_update(stage_t* s, int64_t t, const update_hparams_t* hp) {
  if (!s || !hp) return fail(STAGE_EINVAL, "null argument");
  if (hp->delay < 0 || hp->delay > s->ndelay)
    return fail(STAGE_EINVAL, "delay must be in [0, " + std::to_string(s->ndelay) + "] (the stage's max_delay)");
  if (hp->delay == 0 && hp->ef_lambda != 0.f) return fail(STAGE_EINVAL, "Error Feedback needs a delay >= 1");
  if (int rc = check_update_hparams(hp)) return rc;
  if (hp->optimizer == 1 && s->sh.optimizer != 1)
    return fail(STAGE_EINVAL, "Muon needs a stage shaped with optimizer = 1 (its Newton-Schulz workspace)");
  if (hp->optimizer == 4 && s->sh.optimizer != 2)
    return fail(STAGE_EINVAL, "Adan needs a stage shaped with optimizer = 2 (its two extra state vectors)");
  if (hp->optimizer == 1 && (hp->ns_steps < 1 || hp->ns_steps > 32))
    return fail(STAGE_EINVAL, "ns_steps must be in [1, 32]");
  if (t != s->next_t) return fail(STAGE_ESTATE, "delayed_update: expected t = " + std::to_string(s->next_t));
  const int tau = hp->delay;
  const int64_t gstep = t - tau;  // the gradient this iteration consumes
  bool apply = gstep >= 0;
  int gb = 0;
  if (apply) {
    gb = (int)(gstep % s->ng);
    if (s->grad_step[gb] != gstep || s->grad_count[gb] == 0 || s->grad_consumed[gb])
      return fail(STAGE_ESTATE, "gradient of step " + std::to_string(gstep) + " is not available");
    for (const auto& sl : s->slots)
      if (sl.pending && sl.step == gstep)
        return fail(STAGE_ESTATE, "a microbatch of step " + std::to_string(gstep) + " has not run backward");
  }
  const int vout = (int)((t + 1) % 2);
  for (const auto& sl : s->slots)
    if (sl.pending && sl.step % 2 == vout)
      return fail(STAGE_ESTATE, "a pending microbatch still reads the version being overwritten");
  const int64_t k = s->n_updates + 1;
  // EF once u_{t-tau} exists
  const UpdateScalars hs = update_scalars(hp, k, apply, apply && hp->ef_lambda != 0.f && s->n_updates >= tau);
  // Order the update after the backwards whose gradient it reads (buffer gb) and after the last
  // use of the version it overwrites (parity vout); with no such backward on record, after
  // everything on the stage stream.
  flush_pending(s);  // the previous update's deferred chunks go first
  hipStream_t us = s->ust;
  bool after_all = false;
  if (s->ev_bwd_set[vout]) HIP_OK(hipStreamWaitEvent(us, s->ev_bwd[vout], 0));
  else after_all = true;
  if (apply) {
    if (s->ev_grad_set[gb]) HIP_OK(hipStreamWaitEvent(us, s->ev_grad[gb], 0));
    else after_all = true;
  }
  if (after_all) {
    HIP_OK(hipEventRecord(s->ev_now, s->st));
    HIP_OK(hipStreamWaitEvent(us, s->ev_now, 0));
  }
  // The norm pass runs whether or not clipping is on: it is also the non-finite check (a skipped
  // iteration leaves x, m, v and the EF buffer as they are, and still counts for k)
  const float* clip = nullptr;
  const int* flag = nullptr;
  if (apply) {
    timed(s, STAGE_PROF_NORM, 4.0 * s->n_flat, [&] {
      launch_grad_norm(s->grad[gb], false, s->n_flat, hp->clip_norm, s->upd_norm_part, s->upd_norm_out,
                       s->flag, s->skipped, device_cu_count(), us);
    }, us);
    clip = s->upd_norm_out + 1;
    flag = s->flag;
  }
  // bytes: x, m, v r+w (Lion: no v); g read; shadow write; u_prev r+w with EF (no-op pass: x
  // read, shadow write)
  const double ub = apply ? ((hs.opt == UPD_LION ? 16.0 : 24.0) + 4.0 + (s->bf ? 2.0 : 4.0) +
                             (hp->ef_lambda != 0.f ? 8.0 : 0.0))
                          : (4.0 + (s->bf ? 2.0 : 4.0));
  float* up = hp->ef_lambda != 0.f ? s->u_ring[t % tau] : nullptr;  // tau >= 1 whenever lambda != 0
  if (apply && hp->optimizer == 1) {
    // AdamW on the embedding, the gains and the padding ...
    for (const auto& r : s->adamw_ranges) {
      const int64_t o = r.first;
      timed(s, STAGE_PROF_UPDATE, ub * r.second, [&] {
        launch_fused_update(r.second, s->master + o, s->grad[gb] + o, false, s->m + o, s->v + o,
                            up ? up + o : nullptr, (char*)s->ver[vout] + o * s->esz, s->bf ? 2 : 1, hs, clip,
                            flag, r.second > (1 << 22) ? device_cu_count() : 0, us);
      }, us);
    }
    // ... and Muon on the blocks' weight matrices (Alg. 2): momentum and norms, the normalised
    // wide-orientation copy, Newton-Schulz, the update
    int64_t nm = 0;
    for (const auto& mm : s->muon) nm += (int64_t)mm.rows * mm.cols;
    const int nmat = (int)s->muon.size();
    timed(s, STAGE_PROF_UPDATE, (12.0 + 4.0 + 4.0) * nm, [&] {
      launch_muon_momentum(s->muon_tab, nmat, s->muon_nblk, s->grad[gb], s->m, clip, flag, hp->momentum,
                           s->muon_part, s->muon_norm, us);
      launch_muon_prep(s->muon_tab, nmat, s->muon_ntile, s->m, s->muon_norm, us);
    }, us);
    // quintic Newton-Schulz coefficients of the Muon write-up (Jordan et al., 2024); one timed
    // launch per group, its work the method's flops: ns_steps x 2 nb (2 m^2 n + m^3)
    const float ca = 3.4445f, cb = -4.7750f, cc = 2.0315f;
    for (const auto& gr : s->mgroups) {
      const int m = gr.m, n = gr.n;
      const int64_t mn = (int64_t)m * n, mm2 = (int64_t)m * m;
      const double fl = hp->ns_steps * 2.0 * gr.nb * (2.0 * mm2 * n + (double)mm2 * m);
      if (gr.carry) {
        // X as its hi/lo form S = [hi | lo] from step to step (ping-pong):
        //   A  = hi hi^T                                  (bf16, symmetric: the tiles on and above
        //                                                  the diagonal, mirrored)
        //   Pd = c A A + b A, each column twice: Pd[:, 2k] = Pd[:, 2k + 1] = P[:, k]   (bf16)
        //   S' = form of (Pd Y + a (hi + lo)), Y [2m, n] rows 2k, 2k + 1 = hi_k, lo_k: Y is S
        //        read with row stride n, so Pd Y = P hi + P lo in one product
        //   and X = hi + lo of the last S for the update
        GemmArgs g1[2], g3[2];
        for (int q = 0; q < 2; ++q) {
          g1[q] = gemm(m, m, n, gr.S[q], 2 * n, true, gr.S[q], 2 * n, true, gr.A, m);
          g1[q].batch = gr.nb; g1[q].sA = g1[q].sB = 2 * mn; g1[q].sC = mm2; g1[q].sym = 1;
          g3[q] = gemm(m, n, 2 * m, gr.P, 2 * m, true, gr.S[q], n, false, gr.S[q ^ 1], 2 * n);
          g3[q].epi = GEMM_EPI_NS_SPLIT; g3[q].beta_d = ca; g3[q].D = gr.S[q];
          g3[q].batch = gr.nb; g3[q].sA = 2 * mm2; g3[q].sB = g3[q].sC = g3[q].sD = 2 * mn;
        }
        GemmArgs g2 = gemm(m, m, m, gr.A, m, true, gr.A, m, true, gr.P, 2 * m);
        g2.epi = GEMM_EPI_AXPBY_DUP; g2.alpha = cc; g2.beta_d = cb; g2.D = gr.A; g2.ld_aux = m;
        g2.batch = gr.nb; g2.sA = g2.sB = g2.sD = mm2; g2.sC = 2 * mm2;
        timed(s, STAGE_PROF_NS, fl, [&] {
          launch_muon_split(gr.X[0], gr.S[0], (int64_t)gr.nb * m, n, us);
          for (int it = 0; it < hp->ns_steps; ++it) {
            launch_gemm(true, g1[it % 2], us);
            launch_gemm(true, g2, us);
            launch_gemm(true, g3[it % 2], us);
          }
          launch_muon_join(gr.S[hp->ns_steps % 2], gr.X[0], (int64_t)gr.nb * m, n, us);
        }, us);
      } else if (s->bf) {
        // X in fp32, its products from the hi/lo form S = [hi | lo]:
        //   A  = hi hi^T                                                     (bf16, symmetric)
        //   P  = c A A + b A                                                 (bf16)
        //   X <- P lo + a X, then X <- P hi + X                              (fp32, in place)
        GemmArgs g1 = gemm(m, m, n, gr.S[0], 2 * n, true, gr.S[0], 2 * n, true, gr.A, m);
        g1.batch = gr.nb; g1.sA = g1.sB = 2 * mn; g1.sC = mm2; g1.sym = 1;
        GemmArgs g2 = gemm(m, m, m, gr.A, m, true, gr.A, m, true, gr.P, m);
        g2.epi = GEMM_EPI_AXPBY; g2.alpha = cc; g2.beta_d = cb; g2.D = gr.A;
        g2.batch = gr.nb; g2.sA = g2.sB = g2.sC = g2.sD = mm2;
        GemmArgs g3 = gemm(m, n, m, gr.P, m, true, gr.S[0] + n, 2 * n, false, gr.X[0], n, true, ca);
        g3.batch = gr.nb; g3.sA = mm2; g3.sB = 2 * mn; g3.sC = mn;
        GemmArgs g4 = g3;
        g4.B = gr.S[0];
        g4.beta = 1.f;
        timed(s, STAGE_PROF_NS, fl, [&] {
          launch_muon_split(gr.X[0], gr.S[0], (int64_t)gr.nb * m, n, us);
          for (int it = 0; it < hp->ns_steps; ++it) {
            launch_gemm(true, g1, us);
            launch_gemm(true, g2, us);
            launch_gemm(true, g3, us);
            launch_gemm(true, g4, us);
            if (it + 1 < hp->ns_steps) launch_muon_split(gr.X[0], gr.S[0], (int64_t)gr.nb * m, n, us);
          }
        }, us);
      } else {
        timed(s, STAGE_PROF_NS, fl, [&] {
          for (int it = 0; it < hp->ns_steps; ++it) {
            float* X = gr.X[it % 2];
            float* Xn = gr.X[(it + 1) % 2];
            // A = X X^T;  P = c A A + b A;  X' = P X + a X
            GemmArgs g1 = gemm(m, m, n, X, n, true, X, n, true, gr.A, m);
            g1.batch = gr.nb; g1.sA = g1.sB = mn; g1.sC = mm2;
            GemmArgs g2 = gemm(m, m, m, gr.A, m, true, gr.A, m, true, gr.P, m);
            g2.epi = GEMM_EPI_AXPBY; g2.alpha = cc; g2.beta_d = cb; g2.D = gr.A;
            g2.batch = gr.nb; g2.sA = g2.sB = g2.sC = g2.sD = mm2;
            GemmArgs g3 = gemm(m, n, m, gr.P, m, true, X, n, false, Xn, n);
            g3.epi = GEMM_EPI_AXPBY; g3.alpha = 1.f; g3.beta_d = ca; g3.D = X;
            g3.batch = gr.nb; g3.sA = mm2; g3.sB = g3.sC = g3.sD = mn;
            launch_gemm(false, g1, us);
            launch_gemm(false, g2, us);
            launch_gemm(false, g3, us);
          }
        }, us);
      }
    }
    const bool ef = hs.ef != 0;
    timed(s, STAGE_PROF_UPDATE, (s->esz + 8.0 + 4.0 + s->esz + (up ? 8.0 : 0.0)) * nm, [&] {
      launch_muon_apply(s->bf, s->muon_tab, nmat, s->muon_ntile, s->bf ? 0 : hp->ns_steps % 2, s->master, up, s->ver[vout],
                        flag, hp->lr, hp->weight_decay, hp->update_rms, ef, hp->ef_lambda, us);
    }, us);
  } else if (hs.opt == UPD_ADAN) {
    // x, m, n, d, g_last r+w; g read; the copy written; u_prev r+w with EF
    const double ab = apply ? 40.0 + 4.0 + (s->bf ? 2.0 : 4.0) + (hp->ef_lambda != 0.f ? 8.0 : 0.0)
                            : (4.0 + (s->bf ? 2.0 : 4.0));
    timed(s, STAGE_PROF_UPDATE, ab * s->n_flat, [&] {
      launch_fused_update_adan(s->n_flat, s->master, s->grad[gb], false, s->m, s->v, s->adan_d, s->adan_gl, up,
                               s->ver[vout], s->bf ? 2 : 1, hs, clip, flag, device_cu_count(), us);
    }, us);
  } else {
    // overlap mode 2: one chunk per attention backward the stage runs in a step (of at least 2^16
    // elements, 1024-aligned), launched beside them; otherwise the whole pass now
    const int64_t nchunk = s->overlap == 2
        ? std::min<int64_t>((int64_t)s->sh.n_blocks * s->last_mb, s->n_flat >> 16) : 1;
    if (nchunk > 1) {
      auto& p = s->pend;
      const int64_t per = (s->n_flat / nchunk + 1023) / 1024 * 1024;
      for (int64_t o = 0; o < s->n_flat; o += per) p.chunks.emplace_back(o, std::min(per, s->n_flat - o));
      p.next = 0;
      p.g = s->grad[gb];
      p.up = up;
      p.shadow = s->ver[vout];
      p.hs = hs;
      p.clip = clip;
      p.flag = flag;
      p.bytes = ub;
      p.vout = vout;
      p.gb = gb;
      p.apply = apply;
    } else {
      timed(s, STAGE_PROF_UPDATE, ub * s->n_flat, [&] {
        launch_fused_update(s->n_flat, s->master, s->grad[gb], false, s->m, s->v, up, s->ver[vout],
                            s->bf ? 2 : 1, hs, clip, flag, device_cu_count(), us);
      }, us);
    }
  }
  HIP_OK(hipGetLastError());
  // everything enqueued on the stage stream from here on runs after the update
  HIP_OK(hipEventRecord(s->ev_upd, us));
  if (s->overlap) {
    // only the calls that read what this update wrote, or overwrite what it read, wait for it
    HIP_OK(hipEventRecord(s->ev_upd_v[vout], us));
    s->upd_owed_v[vout] = true;
    if (apply) {
      HIP_OK(hipEventRecord(s->ev_upd_g[gb], us));
      s->upd_owed_g[gb] = true;
    }
    s->upd_owed_all = true;
  } else {
    HIP_OK(hipStreamWaitEvent(s->st, s->ev_upd, 0));
  }
  if (apply) {
    s->grad_consumed[gb] = true;
    s->n_updates = k;
  }
  s->version_step[vout] = t + 1;
  s->next_t = t + 1;
  return STAGE_OK;
}

int delayed_update_flat(int64_t n, float* x, const void* g_prev, int32_t g_is_bf16, float* m, float* v,
                        float* u_prev, void* x_shadow, int32_t shadow_is_bf16, int64_t t,
                        const update_hparams_t* hp, const float* clip_scale_dev, void* hip_stream) {
  if (!hp || n < 0 || t < 0) return fail(STAGE_EINVAL, "bad argument");
  if (hp->delay < 1) return fail(STAGE_EINVAL, "delayed_update_flat implements a delay >= 1");
  if (int rc = check_update_hparams(hp)) return rc;
  if (hp->optimizer == 1) return fail(STAGE_EINVAL, "delayed_update_flat implements the elementwise rules (not Muon)");
  if (hp->optimizer == 4) return fail(STAGE_EINVAL, "Adan keeps two more state vectors: delayed_update_flat_adan");
  if (hp->predict && !x_shadow) return fail(STAGE_EINVAL, "weight prediction writes the compute copy: x_shadow needed");
  if (n == 0) return STAGE_OK;
  if (!x || !g_prev || !m || !v) return fail(STAGE_EINVAL, "null vector");
  if (hp->ef_lambda != 0.f && !u_prev) return fail(STAGE_EINVAL, "Error Feedback needs u_prev");
  if (((uintptr_t)x | (uintptr_t)m | (uintptr_t)v | (uintptr_t)u_prev | (uintptr_t)x_shadow) % 16 ||
      (uintptr_t)g_prev % 8)
    return fail(STAGE_EINVAL, "vectors must be 16-byte aligned (g_prev 8-byte)");
  const int64_t tau = hp->delay;
  const bool apply = t >= tau;
  const UpdateScalars hs = update_scalars(hp, t - tau + 1, apply, hp->ef_lambda != 0.f && t >= 2 * tau);
  launch_fused_update(n, x, g_prev, g_is_bf16 != 0, m, v, hp->ef_lambda != 0.f ? u_prev : nullptr,
                      x_shadow, x_shadow ? (shadow_is_bf16 ? 2 : 1) : 0, hs, clip_scale_dev, nullptr, 0,
                      (hipStream_t)hip_stream);
  HIP_OK(hipGetLastError());
  return STAGE_OK;
}

int stage_resume(stage_t* s, int64_t next_t, int32_t delay) {
  if (!s) return fail(STAGE_EINVAL, "null stage");
  if (next_t < 0) return fail(STAGE_EINVAL, "next_t must be >= 0");
  if (delay < 0 || delay > s->ndelay)
    return fail(STAGE_EINVAL, "delay must be in [0, " + std::to_string(s->ndelay) + "] (the stage's max_delay)");
  if (s->next_t != 0 || s->n_updates != 0) return fail(STAGE_ESTATE, "stage_resume needs a stage that has run no update");
  for (const auto& sl : s->slots)
    if (sl.pending) return fail(STAGE_ESTATE, "stage_resume with a pending microbatch");
  // the gradients of steps next_t - delay .. next_t - 1 wait in their buffers, complete
  for (int j = 0; j < s->ng; ++j) {
    s->grad_step[j] = -1;
    s->grad_count[j] = 0;
    s->grad_consumed[j] = true;
  }
  for (int64_t st = std::max<int64_t>(0, next_t - delay); st < next_t; ++st) {
    const int j = (int)(st % s->ng);
    s->grad_step[j] = st;
    s->grad_count[j] = 1;
    s->grad_consumed[j] = false;
  }
  s->next_t = next_t;
  s->n_updates = delay == 0 ? next_t : std::max<int64_t>(0, next_t - delay);  // gradients consumed so far
  return stage_sync_weights(s);
}

size_t grad_norm_flat_workspace_bytes(void) { return norm_scratch_bytes(); }

int grad_norm_flat(int64_t n, const void* g, int32_t g_is_bf16, float clip_norm, float* out_dev,
                   int32_t* nonfinite_dev, void* workspace, size_t workspace_bytes, void* hip_stream) {
  if (n < 0 || !out_dev) return fail(STAGE_EINVAL, "bad argument");
  if (n > 0 && !g) return fail(STAGE_EINVAL, "null gradient");
  if (!workspace || workspace_bytes < norm_scratch_bytes() || (uintptr_t)workspace % 8)
    return fail(STAGE_EINVAL, "workspace must hold grad_norm_flat_workspace_bytes() bytes, 8-byte aligned");
  if ((uintptr_t)g % (g_is_bf16 ? 8 : 16) || (uintptr_t)out_dev % 4)
    return fail(STAGE_EINVAL, "g must be 16-byte (bf16: 8-byte) aligned");
  launch_grad_norm(g, g_is_bf16 != 0, n, clip_norm, (double*)workspace, out_dev, (int*)nonfinite_dev, nullptr,
                   device_cu_count(), (hipStream_t)hip_stream);
  HIP_OK(hipGetLastError());
  return STAGE_OK;
}

int grad_norm_flat_noalloc(int64_t n, const void* g, int32_t g_is_bf16, float clip_norm, float* out_dev,
                           int32_t* nonfinite_dev, void* hip_stream) {
  if (n < 0 || !out_dev) return fail(STAGE_EINVAL, "bad argument");
  if (n > 0 && !g) return fail(STAGE_EINVAL, "null gradient");
  if ((uintptr_t)g % (g_is_bf16 ? 8 : 16) || (uintptr_t)out_dev % 4)
    return fail(STAGE_EINVAL, "g must be 16-byte (bf16: 8-byte) aligned");
  // the first pass runs min(CUs, capacity) blocks, one partial each: the array's capacity bounds the
  // grid, not n
  const int blocks = device_cu_count();
  if ((size_t)blocks * sizeof(double) > norm_scratch_bytes())
    return fail(STAGE_EINVAL, "grad_norm_flat_noalloc: more partials than its static scratch holds");
  int err = 0;
  double* part = norm_static_scratch(&err);
  if (!part) return fail(STAGE_EHIP, std::string("grad_norm_flat_noalloc: symbol lookup: ") +
                                         hipGetErrorString((hipError_t)err));
  launch_grad_norm(g, g_is_bf16 != 0, n, clip_norm, part, out_dev, (int*)nonfinite_dev, nullptr, blocks,
                   (hipStream_t)hip_stream);
  HIP_OK(hipGetLastError());
  return STAGE_OK;
}

int hbm_stream_copy(void* dst, const void* src, size_t bytes, void* hip_stream) {
  if (bytes % 16 || (uintptr_t)dst % 16 || (uintptr_t)src % 16 || (bytes && (!dst || !src)))
    return fail(STAGE_EINVAL, "hbm_stream_copy: 16-byte aligned pointers and a multiple of 16 bytes");
  launch_stream_copy(dst, src, (int64_t)bytes, (hipStream_t)hip_stream);
  HIP_OK(hipGetLastError());
  return STAGE_OK;
}

int delayed_update_flat_adan(int64_t n, float* x, const void* g_prev, int32_t g_is_bf16, float* m, float* v,
                             float* d, float* g_last, float* u_prev, void* x_shadow, int32_t shadow_is_bf16,
                             int64_t t, const update_hparams_t* hp, const float* clip_scale_dev, void* hip_stream) {
  if (!hp || n < 0 || t < 0) return fail(STAGE_EINVAL, "bad argument");
  if (hp->optimizer != 4) return fail(STAGE_EINVAL, "delayed_update_flat_adan needs optimizer 4 (Adan)");
  if (hp->delay < 1) return fail(STAGE_EINVAL, "delayed_update_flat_adan implements a delay >= 1");
  if (hp->predict) return fail(STAGE_EINVAL, "weight prediction is defined for AdamW only");
  if (n == 0) return STAGE_OK;
  if (!x || !g_prev || !m || !v || !d || !g_last) return fail(STAGE_EINVAL, "null vector");
  if (hp->ef_lambda != 0.f && !u_prev) return fail(STAGE_EINVAL, "Error Feedback needs u_prev");
  if (((uintptr_t)x | (uintptr_t)m | (uintptr_t)v | (uintptr_t)d | (uintptr_t)g_last | (uintptr_t)u_prev |
       (uintptr_t)x_shadow) % 16 || (uintptr_t)g_prev % 8)
    return fail(STAGE_EINVAL, "vectors must be 16-byte aligned (g_prev 8-byte)");
  const int64_t tau = hp->delay;
  const bool apply = t >= tau;
  const UpdateScalars hs = update_scalars(hp, t - tau + 1, apply, hp->ef_lambda != 0.f && t >= 2 * tau);
  launch_fused_update_adan(n, x, g_prev, g_is_bf16 != 0, m, v, d, g_last, hp->ef_lambda != 0.f ? u_prev : nullptr,
                           x_shadow, x_shadow ? (shadow_is_bf16 ? 2 : 1) : 0, hs, clip_scale_dev, nullptr, 0,
                           (hipStream_t)hip_stream);
  HIP_OK(hipGetLastError());
  return STAGE_OK;
}

int stage_embed_indices(stage_t* s, int32_t slot, int32_t* ids, int32_t* counts, int32_t* n_unique) {
  if (!s || !ids || !counts || !n_unique) return fail(STAGE_EINVAL, "null argument");
  if (!s->sh.first_stage) return fail(STAGE_EINVAL, "not a first stage");
  if (slot < 0 || slot >= s->sh.max_inflight) return fail(STAGE_EINVAL, "slot out of range");
  const Slot& sl = s->slots[slot];
  if (sl.step < 0) return fail(STAGE_ESTATE, "slot has not run forward");
  HIP_OK(hipStreamWaitEvent(s->st, sl.ev_sort, 0));
  launch_token_compact(sl.row_start, s->sh.vocab, ids, counts, n_unique, s->st);
  HIP_OK(hipGetLastError());
  return STAGE_OK;
}

int stage_poll_nonfinite(stage_t* s, int64_t* skipped) {
  if (!s) return fail(STAGE_EINVAL, "null stage");
  HIP_OK(hipStreamSynchronize(s->st));
  unsigned long long now = 0;
  HIP_OK(hipMemcpy(&now, s->skipped, 8, hipMemcpyDeviceToHost));
  const unsigned long long d = now - s->skipped_seen;
  s->skipped_seen = now;
  if (skipped) *skipped = (int64_t)d;
  return d ? fail(STAGE_ENONFINITE, "non-finite gradient norm: update skipped") : STAGE_OK;
}

int stage_grad_norm(stage_t* s, int32_t which, float* norm_dev) {
  if (!s || !norm_dev || which < 0 || which >= s->ng) return fail(STAGE_EINVAL, "bad argument");
  launch_grad_norm(s->grad[which], false, s->n_flat, 0.f, s->norm_part, s->norm_out, nullptr, nullptr,
                   device_cu_count(), s->st);
  HIP_OK(hipMemcpyAsync(norm_dev, s->norm_out, 4, hipMemcpyDeviceToDevice, s->st));
  HIP_OK(hipGetLastError());
  return STAGE_OK;
}

int stage_profile_enable(stage_t* s, int32_t on) {
  if (!s) return fail(STAGE_EINVAL, "null stage");
  s->prof_on = on != 0;
  return STAGE_OK;
}

int stage_profile_read(stage_t* s, int32_t cls, double* ms, int64_t* launches, double* work) {
  if (!s || cls < 0 || cls >= STAGE_PROF_NCLASS) return fail(STAGE_EINVAL, "bad argument");
  // every stream a timed launch can be on: an update in flight (overlap mode) records on its own
  HIP_OK(hipStreamSynchronize(s->st));
  for (hipStream_t x : {s->ust, s->wst})
    if (x) HIP_OK(hipStreamSynchronize(x));
  prof_collect(s);
  if (ms) *ms = s->prof_ms[cls];
  if (launches) *launches = s->prof_n[cls];
  if (work) *work = s->prof_work[cls];
  s->prof_ms[cls] = 0.0;
  s->prof_n[cls] = 0;
  s->prof_work[cls] = 0.0;
  return STAGE_OK;
}

void stage_destroy(stage_t* s) {
  if (!s) return;
  (void)hipStreamSynchronize(s->st);
  if (s->ust) (void)hipStreamSynchronize(s->ust);
  if (s->wst) (void)hipStreamSynchronize(s->wst);
  for (auto& r : s->prof_pending) { (void)hipEventDestroy(r.a); (void)hipEventDestroy(r.b); }
  for (auto e : s->prof_free) (void)hipEventDestroy(e);
  for (hipEvent_t e : s->ev_grad)
    if (e) (void)hipEventDestroy(e);
  for (auto& sl : s->slots)
    if (sl.ev_sort) (void)hipEventDestroy(sl.ev_sort);
  for (hipEvent_t e : s->ev_upd_g)
    if (e) (void)hipEventDestroy(e);
  for (hipEvent_t e : s->ev_upd_v)
    if (e) (void)hipEventDestroy(e);
  for (hipEvent_t e : {s->ev_bwd[0], s->ev_bwd[1], s->ev_upd, s->ev_now, s->ev_m2s, s->ev_wjoin, s->ev_wg[0],
                      s->ev_wg[1], s->ev_wg[2], s->ev_wg[3], s->ev_wg[4]})
    if (e) (void)hipEventDestroy(e);
  if (s->ust) (void)hipStreamDestroy(s->ust);
  if (s->wst) (void)hipStreamDestroy(s->wst);
  delete s;
}

}  // extern "C"
