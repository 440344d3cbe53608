// Host-side launchers of the stage's gfx950 kernels (internal to the library).
#pragma once
#include <hip/hip_runtime.h>
#include <cstdint>

// ------------------------------------------------------------------ update (update.hip)
// Elementwise update rules of the fused pass (UpdateScalars::opt)
enum { UPD_ADAMW = 0, UPD_LION = 2, UPD_NADAM = 3, UPD_ADAMW_PREDICT = 4, UPD_ADAN = 5 };
struct UpdateScalars {
  float lr, b1, b2, omb1, omb2, bc1, bc2, eps, wd, lam, one_plus_lam;
  int ef;     // 1: Error-Feedback form this call
  int apply;  // 0: write the compute copy only (no pending gradient)
  int opt = UPD_ADAMW;
  float cg = 0.f, cm = 0.f;      // NAdam: lr (1 - mu_k) / (1 - P_k), lr mu_{k+1} / (1 - P_k mu_{k+1})
  float bc1n = 1.f, bc2n = 1.f;  // prediction: bias corrections of update k + 1
  float b3 = 0.f, omb3 = 0.f, bc3 = 1.f;  // Adan: second-moment weight and its bias correction
  int first = 0;                          // Adan: the first update (the gradient difference is 0)
};
size_t norm_scratch_bytes();
// Device address of the current device's file-scope partial-sum array of the norm (norm_scratch_bytes()
// bytes, looked up once per device); nullptr with *err the HIP error code when the lookup fails.
double* norm_static_scratch(int* err);
// blocks: partial sums (and blocks of the first pass), at most norm_scratch_bytes() / 8; <= 0
// takes that maximum.
void launch_grad_norm(const void* g, bool g_bf16, int64_t n, float clip, double* partial,
                      float* out2, int* flag, unsigned long long* skipped, int blocks, hipStream_t st);
// blocks > 0: a resident grid of that many blocks walks the vector (for a pass that runs beside
// the kernels of another stream); 0: one block per 1024 elements.
void launch_fused_update(int64_t n, float* x, const void* g, bool g_bf16, float* m, float* v,
                         float* up, void* shadow, int shadow_kind, const UpdateScalars& hs,
                         const float* clip, const int* flag, int blocks, hipStream_t st);
// Adan (UPD_ADAN): x, m, n (the v slot), d, g_last, u_prev fp32; blocks as launch_fused_update
void launch_fused_update_adan(int64_t n, float* x, const void* g, bool g_bf16, float* m, float* nn, float* d,
                              float* g_last, float* up, void* shadow, int shadow_kind, const UpdateScalars& hs,
                              const float* clip, const int* flag, int blocks, hipStream_t st);
void launch_cast_copy(int64_t n, const float* src, void* dst, bool dst_bf16, hipStream_t st);
void launch_zero(void* p, int64_t bytes, hipStream_t st);
// bytes a multiple of 16, both pointers 16-byte aligned
void launch_stream_copy(void* dst, const void* src, int64_t bytes, hipStream_t st);

// compute units of the current device (gemm_mfma.hip; cached per device)
int device_cu_count();

// ------------------------------------------------------------------ elementwise (elementwise.hip)
// `bf` selects bf16 storage (else fp32) for every activation / weight pointer of the call.
void launch_embed_gather(bool bf, const int32_t* tok, const void* table, void* x0, int rows, int d,
                         int vocab, hipStream_t st);
void launch_rmsnorm_fwd(bool bf, const void* x, const void* gamma, void* y, float* rstd, int rows,
                        int d, float eps, hipStream_t st);
// dx = resid + rstd * (dn*gamma - xhat * mean(dn*gamma*xhat)); dgamma partial sums into
// partial[p][d]; returns the number of partial rows written (at most one per 16 rows).
constexpr int RMS_CHUNK = 32;
int launch_rmsnorm_bwd(bool bf, const void* dn, const void* x, const float* rstd,
                        const void* gamma, const void* resid, void* dx, float* partial, int rows,
                        int d, hipStream_t st);
// out (+)= the column sums of partial[0 .. nchunks), summed in a fixed order; the rows after
// them are scratch for the first level of the sum.
void launch_colsum_partials(float* partial, int nchunks, int d, float* out, bool accumulate,
                            hipStream_t st);
// rows of d floats the partial buffer of launch_rmsnorm_bwd + launch_colsum_partials needs
inline int64_t rms_partial_rows(int rows) {
  const int64_t p = (rows + 15) / 16;
  return p + (p + 15) / 16;
}
void launch_rope(bool bf, void* qkv, int rows, int seq_len, int n_rot_heads, int head_dim, int ld,
                 const float* cos_t, const float* sin_t, bool inverse, hipStream_t st);
void launch_swiglu_fwd(bool bf, const void* gu, void* z, int rows, int f, hipStream_t st);
// token sort for the embedding gradient: positions sorted by token, stably (equal tokens keep
// ascending positions), tokens outside [0, vocab) keyed as vocab (after every valid one); vocab < 2^17.
// ws: scratch of token_sort_ws_elems(n) int32.  sorted_tok / sorted_pos: n uint32 each.
int64_t token_sort_ws_elems(int n);
void launch_token_sort(const int32_t* tok, int n, int vocab, int32_t* ws, uint32_t* sorted_tok,
                       uint32_t* sorted_pos, hipStream_t st);
void launch_token_runs(const uint32_t* sorted_tok, int n, int vocab, int32_t* row_start,
                       int32_t* ids, int32_t* counts, int32_t* n_unique, hipStream_t st);
// ascending unique ids and their counts from row_start (vocab + 1 entries)
void launch_token_compact(const int32_t* row_start, int vocab, int32_t* ids, int32_t* counts, int32_t* n_unique,
                          hipStream_t st);
void launch_embed_scatter(bool bf, const void* dx0, const uint32_t* sorted_pos,
                          const int32_t* row_start, int vocab, int d, float* de, bool accumulate,
                          hipStream_t st);
// cross-entropy rows of fp32 logits [rows, vocab]: the forward writes lse and the row loss
// lse - z[target]; the backward dlogits = (exp(z - lse) - onehot) * scale (bf16/fp32).  Targets
// outside [0, vocab) give zero loss and zero gradient.
void launch_ce_fwd(const float* logits, const int32_t* targets, int rows, int vocab, float* lse,
                   float* row_loss, hipStream_t st);
void launch_ce_bwd(bool bf, const float* logits, const int32_t* targets, const float* lse, int rows, int vocab,
                   float scale, void* dlogits, hipStream_t st);
void launch_mean(const float* v, int n, float* out, hipStream_t st);

// ------------------------------------------------------------------ GEMM (gemm.hip)
// C[m, n] (+)= sum_k A(m, k) B(n, k).  A(m,k) = a_kmajor ? A[m*lda + k] : A[k*lda + m];
// B(n,k) = b_kmajor ? B[n*ldb + k] : B[k*ldb + n].  Inputs bf16 or fp32 (bf), accumulation fp32.
// out_f32: C is fp32 (beta 0: overwrite, 1: accumulate); else C has the input type.
// resid (input type, leading dimension ldc) is added when non-null.
// ws / ws_elems: optional fp32 workspace; when the output tile grid underfills the chip and K is
// long, an fp32-output product is split over K into partial tiles there and summed in a fixed order.
struct GemmArgs {
  int M, N, K;
  const void* A; int lda; bool a_kmajor;
  const void* B; int ldb; bool b_kmajor;
  void* C; int ldc; bool out_f32; float beta;
  const void* resid;
  float* ws = nullptr; int64_t ws_elems = 0;
  int ksplit = 1;  // set by the launcher
  // epilogue 1 (SwiGLU backward): the product is dz [M, N]; aux holds the saved gate|up
  // pre-activations [M, 2N] (row stride ld_aux) and C receives dgate in columns [0, N) and dup in
  // [N, 2N) (row stride ldc): da = dz b s (1 + a (1 - s)), db = dz a s, s = sigmoid(a).
  // epilogue 2 (RoPE): columns [0, rope_cols) of the bf16 output are rotated in pairs
  // (i, i + hd/2) of each hd-wide head by angle(p, i), p = row mod rope_S (tables [rope_S][hd/2]).
  // epilogue 3 (SwiGLU forward): B is [Wgate; Wup] ([2 glu, K], k-contiguous) and the product is
  // the gate|up pre-activations [M, 2 glu] written to C (ldc = 2 glu) as usual, plus
  // z = silu(gate) * up [M, glu] to out2 (row stride ld_out2).  Requires ldc = 2 glu and
  // ld_out2 = glu (the layouts the SwiGLU kernel of the unfused paths assumes).
  int epi = 0;
  const void* aux = nullptr; int ld_aux = 0;
  const float* rope_cos = nullptr; const float* rope_sin = nullptr;
  int rope_cols = 0, rope_hd = 0, rope_S = 0;
  int glu = 0; void* out2 = nullptr; int ld_out2 = 0;
  // epilogue 4 (attention delta): the product is dO [M, N] (heads of delta_hd columns, rows
  // b * delta_S + i) and aux the attention output O in fp32 of the same layout; besides C, writes
  // delta[(b Hq + h) delta_S + i] = sum over head h's columns of dO O (dO rounded to C's type).
  float* delta = nullptr; int delta_hd = 0, delta_S = 0;
  // epilogue 6 (AXPBY): C = alpha (A B) + beta_d D, D of C's type and layout (leading dim ldc).
  float alpha = 1.f, beta_d = 0.f;
  const void* D = nullptr;
  // batch > 1: `batch` independent products of this shape; operand b starts at A + b sA, B + b sB,
  // C + b sC, D + b sD (elements)
  int batch = 1;
  int64_t sA = 0, sB = 0, sC = 0, sD = 0;
  // sym: the product is symmetric (M == N, plain bf16 output): the direct-to-LDS kernels compute
  // the tiles on and above the diagonal only and write each off-diagonal one also transposed; the
  // other kernels ignore the flag (and compute every tile)
  int sym = 0;
};
constexpr int GEMM_EPI_AXPBY = 6;
// epilogue 7 (AXPBY with duplicated columns): C[r, 2c] = C[r, 2c + 1] = alpha (A B)[r, c] +
// beta_d D[r, c], D of row stride ld_aux, C of row stride ldc (>= 2N).
constexpr int GEMM_EPI_AXPBY_DUP = 7;
// epilogue 8 (hi/lo split): x = (A B)[r, c] + beta_d (D[r, c] + D[r, N + c]) and C receives
// hi = bf16(x) at column c and lo = bf16(x - hi) at N + c; C and D of row stride ldc (>= 2N), D
// holding the same form of the previous x.
constexpr int GEMM_EPI_NS_SPLIT = 8;
// the batched direct-to-LDS kernels take a product (and epilogues 6-8) when it has whole tiles
inline bool gemm_batched_tiles(int M, int N, int K) { return M % 128 == 0 && N % 128 == 0 && K % 64 == 0 && K > 0; }
// y = alpha y + beta x over rows x cols (row stride ld), in place, bf16 or fp32 storage
void launch_axpby(bool bf, void* y, const void* x, float alpha, float beta, int rows, int cols, int ld,
                  hipStream_t st);
constexpr int64_t GEMM_WS_ELEMS = 16 << 20;  // 64 MiB of fp32 split-K partials per stage
void launch_gemm(bool bf, const GemmArgs& g, hipStream_t st);

// ------------------------------------------------------------------ attention (attention.hip)
// Causal grouped-query attention on the packed projection buffer qkv [B*s, (Hq + 2 Hkv) hd]
// (query heads, then key heads, then value heads); o [B*s, Hq hd]; lse fp32 [B, Hq, s].
// rope_cos / rope_sin (backward, optional): qkv holds RoPE-rotated q and k; the returned dq and
// dk are then taken with respect to the unrotated projections (inverse rotation applied).
struct AttnArgs {
  int B, S, Hq, Hkv, hd;
  const void* qkv; void* o; float* lse;
  const void* dout; void* dqkv; float* delta;  // backward only; delta fp32 [B, Hq, s]
  // fp32 copy of o (bf16 stage): the forward writes it when non-null; rowsum(dO O) reads it when
  // non-null (else o)
  float* o32 = nullptr;
  const float* rope_cos = nullptr; const float* rope_sin = nullptr;
  bool delta_ready = false;  // backward: delta already holds rowsum(dO O)
};
void launch_attention_fwd(bool bf, const AttnArgs& a, hipStream_t st);
// delta = rowsum(dO O) per (batch, head, query) alone (O from o32 when set)
void launch_attention_delta(bool bf, const AttnArgs& a, hipStream_t st);
void launch_attention_bwd(bool bf, const AttnArgs& a, hipStream_t st);

// ------------------------------------------------------------------ Muon (muon.hip)
// One weight matrix of delayed Muon: W [rows, cols] row-major at element offset `off` of the flat
// parameter vectors; x[0], x[1] its fp32 Newton-Schulz iterates in wide orientation (the
// transpose, [cols, rows], when trans): ping-pong buffers of the fp32 stage, x[0] alone (updated
// in place) on the bf16 stage; blk0 / tile0 its first block in the element-chunk grid of the
// momentum pass and in the 64 x 64 tile grid of the prep and apply passes.
constexpr int MUON_CHUNK = 4096;
struct MuonMat {
  int64_t off;
  int rows, cols, trans;
  int blk0, tile0;
  float sqrt_max;  // sqrt(max(rows, cols)): the update is scaled to RMS rms with s = rms sqrt_max
  float* x[2];
};
int64_t muon_chunks(int64_t numel);
int64_t muon_tiles(int rows, int cols);
// M <- mu M + (1 - mu) c g on every matrix, then norm[i] = ||M_i||_F (partial: nblk doubles)
void launch_muon_momentum(const MuonMat* mats, int nmat, int nblk, const float* g, float* M, const float* clip,
                          const int* flag, float mu, double* partial, float* norm, hipStream_t st);
// x[0] = M / (||M|| + 1e-7) in wide orientation (fp32)
void launch_muon_prep(const MuonMat* mats, int nmat, int ntile, const float* M, const float* norm, hipStream_t st);
// The bf16 operand form of fp32 iterates X [rows, n] (row stride n): S [rows, 2n] holds, per row,
// [hi | lo] with hi = bf16(x) and lo = bf16(x - hi), so that a product L X is L S[:, 0:n] +
// L S[:, n:2n] (row stride 2n), or one product over K = 2 rows with S read as [2 rows, n] (rows
// 2k, 2k + 1 = hi and lo of row k)
void launch_muon_split(const float* X, bf16* S, int64_t rows, int n, hipStream_t st);
// the inverse: X = hi + lo (n a multiple of 4)
void launch_muon_join(const bf16* S, float* X, int64_t rows, int n, hipStream_t st);
// W, u_prev and the compute copy (bf16 when bf) from O = x[fin]
void launch_muon_apply(bool bf, const MuonMat* mats, int nmat, int ntile, int fin, float* W, float* up,
                       void* shadow, const int* flag, float lr, float wd, float rms, bool ef, float lam,
                       hipStream_t st);

