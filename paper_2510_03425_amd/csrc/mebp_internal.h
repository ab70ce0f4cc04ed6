// Host-side launcher interface between the C-ABI layer (api.hip) and the kernel files.
// Every launcher enqueues on `st` and returns the hipError_t of the launch.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

typedef __bf16 bf16;
typedef _Float16 f16;

namespace mebp {

// ---------------------------------------------------------------- dequant GEMMs
// Forward orientation: C[m][n] = sum_k X[m][k] * W[n][k] with W int4 [N][K/2] + fp16
// scales [N][ceil(K/32)], X fp16 [M][lda] (fp16 MFMA operands). Up to three weight segments along N share X
// (q|k|v, gate|up). Epilogue adds s * u[m][:] . B[n][:] (LoRA up-projection) when
// `lora_B` is set, then the fp32 residual when `resid` is set.
enum NtEpi { NT_STORE_F16 = 0, NT_STORE_F32 = 1, NT_LOGITS = 2 };

struct NtSeg {
  const uint8_t* q4;
  const uint16_t* scale;
  int N;
  int tile0;              // first N-tile index of this segment in the grid (set by the launcher)
  int col0;               // first column of this segment in the split-K partial planes
  const float* lora_u;    // [M][r] (LoRA down-projection output), or null
  const float* lora_B;    // [N][r], or null
  void* out;              // fp16 or fp32 [M][ldo]
  int ldo;
  const float* resid;     // fp32 [M][ldr] added in the epilogue, or null
  int ldr;
  int rope;               // 1: rotate-half RoPE on the (fp16) output, heads of rope_dh columns
  int item0;              // set by the launcher (finalize work-item offset)
};

struct NtArgs {
  const void* X;          // fp16
  int lda, M, K;
  int nseg;
  NtSeg seg[3];
  float lora_s;
  int r;
  // NT_LOGITS: per (row, 64-column tile) the maximum and the sum of exp(logit - max) into
  // `stats` [M][ntiles] float2 (ntiles = row pitch), the logits minus their tile's maximum
  // as fp16 into seg[0].out, and the fp32 logit of the target into tgt_logit[m] (target ids
  // are global vocabulary columns; the segment's first column is vbase).
  float2* stats;
  const int32_t* tgt;     // [M] target id or -1
  float* tgt_logit;
  int ntiles;
  int vbase;
  // split-K scratch (unused when the launcher picks one split)
  float* part;
  size_t part_floats;
  int ldp;                // set by the launcher
  // fused follow-ups, done by the split finalize kernel or, unsplit, by extra kernels:
  const float* rope_cs;   // RoPE table [T][dh/2] (cos, sin) for segments with rope = 1
  int rope_T, rope_dh;
  int gated;              // seg[0] = gate, seg[1] = up: z = act(g) * u into z_out (fp16)
  int act;
  f16* z_out;
  int store_gu;           // gated: also store g and u (fp16) into seg[0].out / seg[1].out
  const float* norm_w;    // single fp32-output segment h: c = fp16(rmsnorm(h) * w) into norm_out
  f16* norm_out;
  float eps;
};
// lora_ready (optional): an event the launch waits on right before the first kernel that
// reads the LoRA factors (the GEMM itself when unsplit, else the split finalize), so that
// the LoRA projection may run on another stream beside the GEMM's main loop.
hipError_t launch_gemm_nt(const NtArgs& a, int epi, hipStream_t st, hipEvent_t lora_ready = nullptr);
int gemm_nt_tiles(int N);  // number of 128-wide N tiles
int gemm_splits(int tiles, int ktiles);
size_t gemm_part_floats(int M, int ncols, int splits);
constexpr int kGemmBM = 128, kGemmBN = 128, kGemmBK = 64;

// Tiling plan: big = 1 selects the 256 x bn tiles of gemm_big.hip (many tokens), else the
// 128 x 128 tiles of gemm_q4.hip; splits = split-K factor before the scratch-capacity check.
struct GemmPlan {
  int big, bn, splits;
};
GemmPlan plan_big(int M, int ntiles256, int ntiles128, int ktiles, bool logits, int max_bn);
GemmPlan plan_nt(int M, const int* Ns, int nseg, int K, int epi);
GemmPlan plan_tn(int M, int Kout, const int* Ns, int nseg, bool softmax);  // softmax: the LM head's dH
// statistics tiles per row of the LM-head logits GEMM over V columns (64 columns each)
int gemm_logit_stat_tiles(int V);
hipError_t launch_gemm_nt_big(const NtArgs& a, int epi, int bn, int S, double flops, double bytes, hipStream_t st);
// whether launch_gemm_nt_big forms z = act(g) * u of a gated product in its epilogue
bool nt_gated_fused(const NtArgs& a, int epi, int bn, int S);

// Transposed orientation (input gradients): C[m][c] = sum_seg sum_n G_seg[m][n] * W_seg[n][c]
// with W_seg int4 [N_seg][Kout/2]; reduction over the weight's output dim; G bf16 (bf16
// MFMA operands).
enum TnEpi { TN_STORE_F32 = 0, TN_ACT_BWD = 1, TN_PARTIAL_F32 = 2, TN_STORE_BF16 = 3 };
enum TnAMode { TN_A_BF16 = 0 };  // the A operand is a bf16 matrix

struct TnSeg {
  const bf16* G;           // [M][ldg]
  int ldg;
  const uint8_t* q4;
  const uint16_t* scale;
  int N;                   // reduction length of this segment
  const float* lora_du;    // [M][r] LoRA gradient du, or null
  const float* lora_A;     // [r][Kout], or null
};

struct TnArgs {
  int M, Kout;
  int nseg;
  TnSeg seg[3];
  int r;
  float* out;              // fp32 [M][ldo] (TN_STORE_F32); partials [splits][M][ldo]
  bf16* outb;              // bf16 [M][ldo] (TN_STORE_BF16)
  int ldo;
  int splits;              // split of the reduction (TN_PARTIAL_F32 only)
  // TN_ACT_BWD: dz -> dg = dz*u*act'(g), du = dz*act(g); fp16 g,u are read and overwritten
  // in place by bf16 dg,du
  void* g;
  void* u;
  int ldgu;
  int act;
  // TN_STORE_BF16 follow-up for the attention backward: delta[b][h][t] = sum_e dO[n][h*dh+e] *
  // delta_o[n][h*dh+e] over the stored bf16 dO (n = b*delta_T + t, O with the same pitch ldo)
  const f16* delta_o;
  float* delta;
  int delta_T, delta_dh;
  // split-K scratch for the stored epilogues (unused with one split)
  float* part;
  size_t part_floats;
  // TN_STORE_F32 follow-up: out2 = resid2 + rmsnorm_bwd(norm_x, norm_w, v), plus a bf16 copy
  const float* norm_x;
  const float* norm_w;
  const float* resid2;
  float* out2;
  bf16* out2b;
  float eps;
  // optional scratch for a transient bf16 copy of the segments' weights: when the large-tile
  // kernel is chosen and sum_seg N_seg * Kout <= w16_elems, the weights are decompressed
  // into it first (bf16 of q * s, rounded to nearest even, [N_seg][Kout] back to back) and
  // the kernel reads them without decompressing (identical operands, identical results)
  uint16_t* w16;
  size_t w16_elems;
};
hipError_t launch_gemm_tn(const TnArgs& a, int epi, int amode, hipStream_t st, hipEvent_t lora_ready = nullptr);
// w16: seg.q4 points at bf16 weights [N][Kout] (no scales)
hipError_t launch_gemm_tn_big(const TnArgs& a, int epi, int amode, int bn, int S, double flops, double bytes,
                              hipStream_t st, bool w16 = false);
// bf16 elements of the transient weight copy that launch_gemm_tn would use for these
// segments (0 when the large-tile kernel is not chosen)
size_t gemm_tn_w16_elems(int M, int Kout, const int* Ns, int nseg, bool softmax);

// Test aid: one production GEMM kernel chosen by `kind` (the MEBP_TEST_GEMM_* values of the
// C ABI) on caller operands, one split, no LoRA term or residual, fp32 outputs. Forward
// kinds: out[M][n_out] = X fp16 [M][n_in] times W^T; transposed kinds: out[M][n_in] =
// G bf16 [M][n_out] times W. launch_gemm_probe handles the 128 x 128 kernels and hands the
// large-tile kinds to launch_gemm_probe_big.
hipError_t launch_gemm_probe(int kind, const uint8_t* q4, const uint16_t* scale, int n_out, int n_in, const void* x,
                             int M, float* out, hipStream_t st);
hipError_t launch_gemm_probe_big(int kind, const uint8_t* q4, const uint16_t* scale, int n_out, int n_in,
                                 const void* x, int M, float* out, hipStream_t st);

// ---------------------------------------------------------------- elementwise / norms
hipError_t launch_dequant(const uint8_t* q4, const uint16_t* scale, int rows, int cols, int group,
                          float* out_f32, uint16_t* out_bf16, hipStream_t st);
hipError_t launch_embed(const uint8_t* q4, const uint16_t* scale, int d, int group, const int32_t* ids,
                        int n, int V, float* x0, hipStream_t st, float mul = 1.0f);
// out = resid + RMSNorm(t) * w (row-wise)
hipError_t launch_resid_rmsnorm(const float* resid, const float* t, const float* w, int n, int d, float eps,
                                float* out, hipStream_t st);
// in place on fp16 q or k heads [n][ld]: + bias (if any), per-head RMSNorm with weight nw (if
// any; pre-norm values to `pre`, same layout), RoPE (if rope); for v: bias only
hipError_t launch_qkv_post(f16* x, int ld, int n, int T, int H, int dh, const float* bias, const float* nw, float eps,
                           f16* pre, const float* cs, int rope, hipStream_t st);
// per-head RMSNorm backward in place on bf16 g [n][ldg] from pre-norm values pre [n][ld]
hipError_t launch_headnorm_bwd(const f16* pre, int ld, int n, int H, int dh, const float* nw, float eps, bf16* g,
                               int ldg, hipStream_t st);
// y = fp16(x * w * rstd); rstd optional
hipError_t launch_rmsnorm_fwd(const float* x, const float* w, int n, int d, float eps, f16* y,
                              float* rstd, hipStream_t st);
// dx = resid + rmsnorm_bwd(x, w, dy); writes fp32 dx (may alias resid) and optional bf16 copy
hipError_t launch_rmsnorm_bwd(const float* x, const float* w, const float* dy, const float* resid,
                              int n, int d, float eps, float* dx, bf16* dx_bf16, hipStream_t st);
hipError_t launch_f32_to_bf16(const float* x, bf16* y, size_t n, hipStream_t st);
hipError_t launch_rope_table(int T, int dh, double theta, float* cs, hipStream_t st);
// in-place rotate-half RoPE on fp16 rows [B*T][H*dh] (columns head-major)
hipError_t launch_rope_fwd(f16* x, int ld, int B, int T, int H, int dh, const float* cs, hipStream_t st);
hipError_t launch_act_fwd(const f16* g, const f16* u, f16* z, size_t n, int act, hipStream_t st);

// ---------------------------------------------------------------- LoRA skinny kernels
// Split scratch: fp32 partial planes of split reductions (LoRA outer, attention dK/dV).
struct SplitScratch {
  float* part;
  size_t part_floats;
};
// Rows: out[m][j] = s * sum_k X[m][k] * W(j, k) for each job, W(j,k) = W[j*K + k]
// (wt = 0, A [r][K]) or W[k*r + j] (wt = 1, B [K][r]); X [M][ldx], fp16 (xbf16 = 0) or
// bf16 (xbf16 = 1), the same type for every job of a launch.
struct LoraRowsJob {
  const void* X;
  int ldx, K;
  const float* W;
  float* out;             // [M][r]
};
struct LoraRowsArgs {
  LoraRowsJob job[3];
  int njobs, M, r, wt;
  float s;
};
hipError_t launch_lora_rows(const LoraRowsArgs& a, int xbf16, hipStream_t st);
// Outer: R(c, j) = s_job * sum_m Mx[m][c] * V[m][j] for each job, written as out[c*r + j]
// (layout 0, dB [C][r]) or out[j*C + c] (layout 1, dA [r][C]). Mx [M][ldm] fp16 (mbf16 = 0)
// or bf16 (mbf16 = 1), V fp32 [M][r]. Token-split partials use `part` when the token count
// is large (lora_outer_part_floats).
struct LoraOuterJob {
  const void* Mx;
  int ldm, C;
  const float* V;
  float* out;
  float s;
};
struct LoraOuterArgs {
  LoraOuterJob job[3];
  int njobs, M, r, layout;
  float* part;
  size_t part_floats;
  int cmax;               // set by the launcher
};
hipError_t launch_lora_outer(const LoraOuterArgs& a, int mbf16, hipStream_t st);
size_t lora_outer_part_floats(int M, int cmax, int r, int njobs);
hipError_t launch_fill_i32(int* p, int n, int v, hipStream_t st);

// ---------------------------------------------------------------- attention
struct AttnArgs {
  const f16* q; const f16* k; const f16* v;      // [B*T][H*dh] row-major, head-major cols
  int ldq, ldk;                                  // row pitch of q (Hq*dh) and k/v (Hkv*dh)
  int B, T, Hq, Hkv, dh, window;
  f16* o;                                        // [B*T][Hq*dh]
  float* lse;                                    // [B][Hq][T]
  // backward
  const bf16* dO; const float* delta;            // delta [B][Hq][T]
  const float* cs;                               // rope table of this layer [T][dh/2][2]
  bf16* dq; bf16* dk; bf16* dv;                  // gradients (dq, dk pre-RoPE)
};
// Launch plan of one attention shape: which forward kernel, and the chunking of the
// forward / dQ key loops and the dK/dV query loop when the tile grid alone would leave
// compute units idle (0 chunks = no split). Scratch floats: forward chunk partials; dK/dV
// partials (grouped-query heads and/or chunks); dQ chunk partials (after the dK/dV ones).
struct AttnPlan {
  bool fwd32;
  int f_nck, f_ck, q_nck, q_ck, kv_nck, kv_cq;
  size_t fwd_floats, kv_floats, q_floats;
};
AttnPlan attn_plan(int B, int T, int Hq, int Hkv, int dh, int window);
// split scratch the attention of this shape needs (forward and backward use it at
// different times)
size_t attn_part_floats(int B, int T, int Hq, int Hkv, int dh, int window);
hipError_t launch_attn_fwd(const AttnArgs& a, const SplitScratch& sc, hipStream_t st);
// scratch: delta [B][Hq][T], and the partials of attn_plan in sc.
// With `aux` (and two events), the dQ kernels run there beside dK/dV; `st` waits for them
// before returning.
// delta_ready: delta_ws already holds rowsum(dO * O) (computed with dO, see TnArgs::delta).
hipError_t launch_attn_bwd(const AttnArgs& a, float* delta_ws, const SplitScratch& sc, hipStream_t st,
                           hipStream_t aux = nullptr, hipEvent_t ev_go = nullptr, hipEvent_t ev_done = nullptr,
                           bool delta_ready = false);
// delta[b][h][t] = sum_e dO[b*T+t][h*dh+e] * O[b*T+t][h*dh+e] (rows of pitch ld)
hipError_t launch_attn_delta(const bf16* dO, const f16* O, int ld, int B, int T, int H, int dh, float* delta,
                             hipStream_t st);

// ---------------------------------------------------------------- optimizer
// One LoRA tensor of an elementwise optimizer launch: n4 float4s at p (updated), g (read),
// m, v (AdamW moments, updated; unused by accumulation). All 16-byte aligned.
struct OptSeg {
  float* p; const float* g; float* m; float* v;
  uint32_t n4;
};
constexpr int OPT_MAXSEG = 80;  // keeps OptArgs (a kernel argument) under 4 KB
struct OptArgs {
  OptSeg seg[OPT_MAXSEG];
  uint32_t blk0[OPT_MAXSEG];  // first workgroup of each segment
  int nseg;
  float lr, beta1, beta2, eps, weight_decay, inv_bc1, inv_bc2, grad_scale;
};
// mode 0: AdamW with the parameters in `a`; mode 1: p = (first ? 0 : p) + scale * g.
hipError_t launch_lora_opt(const OptSeg* segs, int nseg, OptArgs a, int mode, float scale, int first,
                           hipStream_t st);

// ---------------------------------------------------------------- LM head / CE
// The vocabulary is processed in chunks of columns [v0, v0 + w) (see k_ce_* in
// elementwise.hip): running per-row maximum m and sum l, a rescaled fp32 dH accumulator.
// chunk statistics from the logits GEMM's per-(row, 64-column tile) (max, sum exp) into
// the running (m, l); alpha = exp(m_old - m_new)
hipError_t launch_ce_chunk_stats(const float2* stats, int ld, int nt, int M, float* mrun, float* lrun, float* alpha,
                                 int first, hipStream_t st);
// in place: tile-relative fp16 logits of the chunk -> bf16 exp(logit - m), 0 at the target
// column and on rows without a target
hipError_t launch_ce_probs(uint16_t* logits, int M, int w, int ld, const float2* stats, int ld_tiles,
                           const float* mrun, const int32_t* tgt, int v0, hipStream_t st);
// dh = (first ? 0 : alpha[m] dh) + sum of the chunk product's split planes
hipError_t launch_ce_dh_accum(const float* part, int splits, int M, int d, const float* alpha, int first, float* dh,
                              hipStream_t st);
// lse, row loss terms, and dhf = inv_n (dh / l + (P_target - 1) E[target]) in place
hipError_t launch_ce_final(int M, int d, const uint8_t* eq4, const uint16_t* escale, const int32_t* tgt,
                           const float* tgt_logit, const float* mrun, const float* lrun, float inv_n, float* dhf,
                           float* lse, float* row_loss, hipStream_t st);
hipError_t launch_ce_loss(const float* row_loss, const int32_t* tgt, int M, float inv_n, float* loss,
                          hipStream_t st);
// bytes (a multiple of 16) between device memory and pinned host memory addressed through
// its device address (both 16-byte aligned), by a few workgroups on `st`
hipError_t launch_copy_host(const void* src, void* dst, size_t bytes, hipStream_t st);
hipError_t launch_targets(const int32_t* ids, int B, int T, int V, int32_t* tgt, hipStream_t st);

// ---------------------------------------------------------------- diagnostics
// Per-kernel event timing (see timing.hip). timer_begin returns -1 when disabled.
// count: launches bracketed by this record (a repeated burst counts as `count` launches)
int timer_begin(hipStream_t st, const char* name, double flops, double bytes, int count);
void timer_end(hipStream_t st, int token);
int timing_enable(int enable, int capacity);
int timing_report(char* buf, size_t len);
int repeat_count(const char* name);
int set_repeat(const char* name, int times);

// Bracket one launch statement (issued repeat_count times back to back) with the
// optional timer.
#define MEBP_TIMED(st, name, flops, bytes, stmt)                                  \
  do {                                                                            \
    const char* name_ = (name);                                                   \
    const int reps_ = ::mebp::repeat_count(name_);                                \
    const int tok_ = ::mebp::timer_begin((st), name_, (flops), (bytes), reps_);   \
    for (int rep_ = reps_; rep_ > 0; --rep_) {                                    \
      stmt;                                                                       \
    }                                                                             \
    ::mebp::timer_end((st), tok_);                                                \
  } while (0)

}  // namespace mebp
