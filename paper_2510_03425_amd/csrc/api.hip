// C ABI of libmebp: argument validation, workspace layout and the orchestration of the
// checkpointed LoRA step (Algorithm 1) out of the gfx950 kernels. Every entry point
// validates everything before enqueuing anything; nothing here allocates device memory.
#include <math.h>
#include <stdlib.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <atomic>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#define MEBP_RING_MAX 16

#include "../../include/mebp.h"
#include "mebp_internal.h"

using namespace mebp;

// Scratch of mebp_layer_recompute_backward_static: one copy per device, reserved with the
// library's code object. In host code this name is only a handle for the runtime's symbol
// lookup, never an address (see static_scratch()).
static __device__ __attribute__((aligned(256))) uint8_t scratch[MEBP_STATIC_SCRATCH_BYTES];

namespace {

thread_local std::string g_last_error;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return code;
}

#define HIP_TRY(expr)                                                                  \
  do {                                                                                 \
    hipError_t e_ = (expr);                                                            \
    if (e_ != hipSuccess) return fail(MEBP_EHIP, "%s: %s", #expr, hipGetErrorString(e_)); \
  } while (0)

bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

// ------------------------------------------------------------------ workspace layout
enum Slot {
  S_A, S_Q, S_K, S_V, S_O, S_LSE, S_H, S_C, S_G, S_U, S_Z, S_LU, S_LDU, S_DYB, S_DC, S_DH, S_DHB, S_DO,
  S_DELTA, S_DQ, S_DK, S_DV, S_DA, S_PART, S_ROPE_G, S_ROPE_L, S_TGT, S_HF, S_LOGITS, S_STATS, S_LSEV,
  S_TGTLOGIT, S_ROWLOSS, S_DHF, S_LMPART, S_GRAD, S_SPLIT, S_QPRE, S_KPRE, S_TO, S_TD, S_DTB, S_DTOB, S_CEMAX,
  S_CESUM, S_CEALPHA, S_W16, S_COUNT
};
const char* kSlotNames[S_COUNT] = {
  "a", "q", "k", "v", "o", "lse", "h", "c", "g", "u", "z", "lora_u", "lora_du", "dy_bf16", "dc", "dh",
  "dh_bf16", "do", "delta", "dq", "dk", "dv", "da", "lora_part", "rope_global", "rope_local", "targets",
  "hf", "logits", "ce_stats", "ce_lse", "ce_target_logit", "ce_row_loss", "dhf", "lm_part", "grad", "split_part",
  "q_prenorm", "k_prenorm", "attn_out_prenorm", "mlp_out_prenorm", "d_mlp_out_bf16", "d_attn_out_bf16", "ce_max",
  "ce_sum", "ce_alpha", "w16"};

// Slots written by a layer's (re)computed forward and read by its backward, plus the
// split-K scratch: the training step keeps two copies, so that the recompute of layer l-1
// (on the side stream) can run while layer l is backpropagated. The bf16 copy of the
// upstream gradient alternates too: layer l reads its set's copy and writes bf16(dx) into
// the other one, which the LoRA gradient kernels of layer l may still be reading from.
bool per_set(int s) {
  switch (s) {
    case S_A: case S_Q: case S_K: case S_V: case S_O: case S_LSE: case S_H: case S_C: case S_G: case S_U:
    case S_Z: case S_LU: case S_DYB: case S_SPLIT: case S_QPRE: case S_KPRE: case S_TO: case S_TD:
      return true;
    default:
      return false;
  }
}

// Debug mode of the workspace (mebp_set_workspace_guards, or MEBP_WS_GUARD=1 in the
// environment when the library loads): every slot, both copies of the per-set ones, is
// followed by a guard region (its padding up to the 256-byte boundary plus 256 bytes) that
// holds a known pattern. The entry points that take a workspace fill the guards before
// their first kernel and check them after their last one on the caller's stream, then wait
// for the stream: an overwritten guard fails the call with MEBP_EWORKSPACE and the slot's
// name. The layout, and so mebp_workspace_bytes, depends on the mode.
std::atomic<int> g_guards{[] {
  const char* e = getenv("MEBP_WS_GUARD");
  return e && *e && *e != '0' ? 1 : 0;
}()};
constexpr size_t kGuardBytes = 256;
constexpr int kMaxGuards = 2 * S_COUNT;

struct Layout {
  size_t off[S_COUNT];
  size_t off1[S_COUNT];  // second copy of the per-set slots (equal to off[] for the others)
  size_t total;
  bool guards;                // debug mode: guard regions after the slots
  int nguard;
  size_t g_off[kMaxGuards];   // guard regions: byte offset, length (multiples of 4) and
  uint32_t g_len[kMaxGuards]; // tag = slot + S_COUNT * copy
  int32_t g_tag[kMaxGuards];
  size_t status_off;          // one word: the smallest tag of an overwritten guard
  int lm_chunk;   // vocabulary columns per LM-head chunk
  int lm_splits;  // split-K factor of a whole chunk's dH product (narrower chunks use fewer)
  int ntiles;     // statistics tiles of a whole chunk (the stats row pitch)
  size_t split_floats;
  size_t lora_part_floats;
  size_t w16_elems;  // transient bf16 weights of the large-tile transposed products
};

size_t nt_part(int M, int K, std::initializer_list<int> Ns) {
  int v[3], n = 0, ncat = 0;
  for (int x : Ns) {
    v[n++] = x;
    ncat += x;
  }
  return gemm_part_floats(M, ncat, plan_nt(M, v, n, K, NT_STORE_F32).splits);
}
size_t tn_part(int M, int Kout, std::initializer_list<int> Ns) {
  int v[3], n = 0;
  for (int x : Ns) v[n++] = x;
  return gemm_part_floats(M, Kout, plan_tn(M, Kout, v, n, false).splits);
}

// Columns of one LM-head vocabulary chunk: the chunk's fp16 logits [N][chunk] take at most
// MEBP_LM_CHUNK_MB (default 512) MiB; a multiple of 256 columns, the whole vocabulary when
// it fits.
int lm_chunk_cols(size_t N, int V) {
  static const size_t budget = [] {
    const char* e = getenv("MEBP_LM_CHUNK_MB");
    const long v = e && *e ? atol(e) : 512;
    return (size_t)(v > 0 ? v : 512) << 20;
  }();
  size_t c = budget / (N * 2) / 256 * 256;
  if (c < 256) c = 256;
  return c >= (size_t)V ? V : (int)c;
}

int lm_head_splits(int N, int d, int V) {
  // token tiles are 256 rows in the large-tile kernel, 128 in the other
  const int bm = plan_tn(N, d, &V, 1, true).big ? 256 : 128;
  const int tiles = ((d + 127) / 128) * ((N + bm - 1) / bm);
  int s = (512 + tiles - 1) / tiles;
  const int max_s = ((V + 63) / 64 + 7) / 8;
  if (s > max_s) s = max_s;
  if (s > 64) s = 64;
  if (s < 1) s = 1;
  return s;
}

bool make_layout(const mebp_config* c, int B, int T, Layout* L) {
  const size_t N = (size_t)B * T, d = c->hidden, qd = (size_t)c->n_heads * c->head_dim,
               kvd = (size_t)c->n_kv_heads * c->head_dim, F = c->ffn, r = c->lora_rank > 0 ? c->lora_rank : 16,
               V = c->vocab, H = c->n_heads;
  L->lm_chunk = V ? lm_chunk_cols(N, (int)V) : 0;
  const size_t Vc = L->lm_chunk;
  L->lm_splits = V ? lm_head_splits((int)N, (int)d, (int)Vc) : 0;
  L->ntiles = V ? gemm_logit_stat_tiles((int)Vc) : 0;
  size_t sz[S_COUNT] = {};
  sz[S_A] = N * d * 2;
  sz[S_Q] = N * qd * 2;
  sz[S_K] = N * kvd * 2;
  sz[S_V] = N * kvd * 2;
  sz[S_O] = N * qd * 2;
  sz[S_LSE] = N * H * 4;
  sz[S_H] = N * d * 4;
  sz[S_C] = N * d * 2;
  sz[S_G] = N * F * 2;
  sz[S_U] = N * F * 2;
  sz[S_Z] = N * F * 2;
  sz[S_LU] = MEBP_NPROJ * N * r * 4;
  sz[S_LDU] = MEBP_NPROJ * N * r * 4;
  sz[S_DYB] = N * d * 2;
  sz[S_DC] = N * d * 4;
  sz[S_DH] = N * d * 4;
  sz[S_DHB] = N * d * 2;
  sz[S_DO] = N * qd * 2;
  sz[S_DELTA] = N * H * 4;
  sz[S_DQ] = N * qd * 2;
  sz[S_DK] = N * kvd * 2;
  sz[S_DV] = N * kvd * 2;
  sz[S_DA] = N * d * 4;
  sz[S_PART] = 0;  // LoRA dA / dB token-split partials (sized below)
  sz[S_ROPE_G] = (size_t)T * c->head_dim * 4;
  sz[S_ROPE_L] = (size_t)T * c->head_dim * 4;
  sz[S_TGT] = N * 4;
  sz[S_HF] = V ? N * d * 2 : 0;
  sz[S_LOGITS] = N * Vc * 2;
  sz[S_STATS] = N * (size_t)L->ntiles * 8;
  sz[S_LSEV] = V ? N * 4 : 0;
  sz[S_TGTLOGIT] = V ? N * 4 : 0;
  sz[S_ROWLOSS] = V ? N * 4 : 0;
  sz[S_DHF] = V ? N * d * 4 : 0;
  sz[S_LMPART] = (size_t)L->lm_splits * N * d * 4;
  sz[S_GRAD] = N * d * 4;
  sz[S_CEMAX] = V ? N * 4 : 0;
  sz[S_CESUM] = V ? N * 4 : 0;
  sz[S_CEALPHA] = V ? N * 4 : 0;
  const bool qkn = c->arch & MEBP_ARCH_QK_NORM, sw = c->arch & MEBP_ARCH_SANDWICH;
  sz[S_QPRE] = qkn ? N * qd * 2 : 0;
  sz[S_KPRE] = qkn ? N * kvd * 2 : 0;
  sz[S_TO] = sw ? N * d * 4 : 0;
  sz[S_TD] = sw ? N * d * 4 : 0;
  sz[S_DTB] = sw ? N * d * 2 : 0;
  sz[S_DTOB] = sw ? N * d * 2 : 0;
  {
    const int M = (int)N, D = (int)d, Q = (int)qd, KV = (int)kvd, FF = (int)F, R = (int)r;
    size_t m = 0;
    auto mx = [&](size_t v) { m = v > m ? v : m; };
    mx(nt_part(M, D, {Q, KV, KV}));
    mx(nt_part(M, Q, {D}));
    mx(nt_part(M, D, {FF, FF}));
    mx(nt_part(M, FF, {D}));
    mx(tn_part(M, FF, {D}));
    mx(tn_part(M, D, {FF, FF}));
    mx(tn_part(M, Q, {D}));
    mx(tn_part(M, D, {Q, KV, KV}));
    // attention scratch for the sliding-window layers and the global ones
    mx(attn_part_floats(B, T, c->n_heads, c->n_kv_heads, c->head_dim, c->window));
    mx(attn_part_floats(B, T, c->n_heads, c->n_kv_heads, c->head_dim, 0));
    L->split_floats = m;
    sz[S_SPLIT] = m * 4;
    // every dB / dA launch of a layer: (widest column count, jobs)
    size_t lp = 0;
    for (size_t v : {lora_outer_part_floats(M, Q > KV ? Q : KV, R, 3), lora_outer_part_floats(M, D, R, 3),
                     lora_outer_part_floats(M, D, R, 1), lora_outer_part_floats(M, Q, R, 1),
                     lora_outer_part_floats(M, FF, R, 2), lora_outer_part_floats(M, D, R, 2),
                     lora_outer_part_floats(M, FF, R, 1)})
      lp = v > lp ? v : lp;
    L->lora_part_floats = lp;
    sz[S_PART] = lp * 4;
    // the transposed products of the backward (down, gate + up, o, q + k + v) and the LM
    // head's dH product over one vocabulary chunk, one at a time
    size_t w = 0;
    const int n_down[1] = {D}, n_gu[2] = {FF, FF}, n_o[1] = {D}, n_qkv[3] = {Q, KV, KV}, n_lm[1] = {(int)Vc};
    for (size_t v : {gemm_tn_w16_elems(M, FF, n_down, 1, false), gemm_tn_w16_elems(M, D, n_gu, 2, false),
                     gemm_tn_w16_elems(M, Q, n_o, 1, false), gemm_tn_w16_elems(M, D, n_qkv, 3, false),
                     V ? gemm_tn_w16_elems(M, D, n_lm, 1, true) : (size_t)0})
      w = v > w ? v : w;
    L->w16_elems = w;
    sz[S_W16] = w * 2;
  }
  size_t o = 0;
  L->guards = g_guards.load() != 0;
  L->nguard = 0;
  auto place = [&](int i, int copy) {
    const size_t at = o;
    o += ((sz[i] + 255) & ~(size_t)255) + (L->guards ? kGuardBytes : 0);
    if (L->guards) {
      const size_t g = at + ((sz[i] + 3) & ~(size_t)3);
      L->g_off[L->nguard] = g;
      L->g_len[L->nguard] = (uint32_t)(o - g);
      L->g_tag[L->nguard] = i + S_COUNT * copy;
      ++L->nguard;
    }
    return at;
  };
  for (int i = 0; i < S_COUNT; ++i) L->off[i] = place(i, 0);
  for (int i = 0; i < S_COUNT; ++i) L->off1[i] = per_set(i) ? place(i, 1) : L->off[i];
  L->status_off = o;
  if (L->guards) o += 256;
  L->total = o;
  return true;
}

template <class Tp>
Tp* slot(void* ws, const Layout& L, int s) {
  return (Tp*)((char*)ws + L.off[s]);
}

// ------------------------------------------------------------------ workspace guards
struct GuardList {
  int n;
  uint32_t len[kMaxGuards];
  int32_t tag[kMaxGuards];
  unsigned long long off[kMaxGuards];
};

__device__ uint32_t guard_word(int32_t tag, uint32_t i) {
  return 0xA5C3E1F7u ^ ((uint32_t)tag * 0x9E3779B9u) ^ (i * 0x85EBCA6Bu);
}

// one block per guard region
__global__ void k_guard_fill(uint8_t* ws, GuardList g) {
  const int r = blockIdx.x;
  uint32_t* p = (uint32_t*)(ws + g.off[r]);
  for (uint32_t i = threadIdx.x; i < g.len[r] / 4; i += blockDim.x) p[i] = guard_word(g.tag[r], i);
}

__global__ void k_guard_reset(uint32_t* status) { *status = 0xFFFFFFFFu; }

__global__ void k_guard_check(const uint8_t* ws, GuardList g, uint32_t* status) {
  const int r = blockIdx.x;
  const uint32_t* p = (const uint32_t*)(ws + g.off[r]);
  bool bad = false;
  for (uint32_t i = threadIdx.x; i < g.len[r] / 4; i += blockDim.x) bad |= p[i] != guard_word(g.tag[r], i);
  if (bad) atomicMin(status, (uint32_t)g.tag[r]);
}

int guard_launch(const Layout& L, void* ws, hipStream_t st, bool fill) {
  GuardList g;
  g.n = L.nguard;
  for (int i = 0; i < L.nguard; ++i) {
    g.off[i] = L.g_off[i];
    g.len[i] = L.g_len[i];
    g.tag[i] = L.g_tag[i];
  }
  uint32_t* status = (uint32_t*)((char*)ws + L.status_off);
  if (fill) {
    hipLaunchKernelGGL(k_guard_fill, dim3(g.n), dim3(128), 0, st, (uint8_t*)ws, g);
  } else {
    // a check may follow another check: the status word starts over
    hipLaunchKernelGGL(k_guard_reset, dim3(1), dim3(1), 0, st, status);
    hipLaunchKernelGGL(k_guard_check, dim3(g.n), dim3(128), 0, st, (const uint8_t*)ws, g, status);
  }
  HIP_TRY(hipGetLastError());
  return MEBP_OK;
}

// Checks every guard on `st` and waits for it: MEBP_EWORKSPACE names the first slot (in
// layout order) whose guard no longer holds its pattern.
int guard_verdict(const Layout& L, void* ws, hipStream_t st) {
  int e = guard_launch(L, ws, st, false);
  if (e) return e;
  uint32_t h = 0;
  HIP_TRY(hipMemcpyAsync(&h, (char*)ws + L.status_off, 4, hipMemcpyDeviceToHost, st));
  HIP_TRY(hipStreamSynchronize(st));
  if (h != 0xFFFFFFFFu)
    return fail(MEBP_EWORKSPACE, "workspace guard after slot '%s'%s was overwritten", kSlotNames[h % S_COUNT],
                h >= (uint32_t)S_COUNT ? " (second copy)" : "");
  return MEBP_OK;
}

// Runs `body` (the launches of one entry point on `stream`) between a fill and a check of
// the guards when the layout has them; otherwise just runs it.
template <class F>
int guarded(const mebp_config* c, int B, int T, void* ws, mebp_stream_t stream, F&& body) {
  if (!g_guards.load()) return body();
  Layout L;
  make_layout(c, B, T, &L);
  if (!L.guards) return body();
  int e = guard_launch(L, ws, (hipStream_t)stream, true);
  if (e || (e = body())) return e;
  return guard_verdict(L, ws, (hipStream_t)stream);
}

// ------------------------------------------------------------------ validation
int check_config(const mebp_config* c) {
  if (!c) return fail(MEBP_EINVAL, "cfg is NULL");
  if (c->n_layers < 1 || c->hidden <= 0 || c->n_heads <= 0 || c->n_kv_heads <= 0 || c->ffn <= 0 || c->vocab < 0)
    return fail(MEBP_EINVAL, "non-positive dimension in config");
  if (c->n_heads % c->n_kv_heads) return fail(MEBP_EINVAL, "n_heads %% n_kv_heads != 0");
  if (c->head_dim != 64 && c->head_dim != 128 && c->head_dim != 256)
    return fail(MEBP_EUNSUPPORTED, "head_dim %d not in {64, 128, 256}", c->head_dim);
  if (c->hidden % 32) return fail(MEBP_EUNSUPPORTED, "hidden %d not a multiple of 32", c->hidden);
  if (c->ffn % 16) return fail(MEBP_EUNSUPPORTED, "ffn %d not a multiple of 16", c->ffn);
  if (c->vocab % 32) return fail(MEBP_EUNSUPPORTED, "vocab %d not a multiple of 32", c->vocab);
  if (c->group != 32) return fail(MEBP_EUNSUPPORTED, "group %d != 32", c->group);
  if (c->act != 0 && c->act != 1) return fail(MEBP_EINVAL, "act %d not 0 (SiLU) or 1 (GELU-tanh)", c->act);
  if (!(c->rms_eps >= 0.f) || !isfinite(c->rms_eps)) return fail(MEBP_EINVAL, "bad rms_eps");
  if (!(c->rope_theta_global > 0.f) || !(c->rope_theta_local > 0.f)) return fail(MEBP_EINVAL, "bad rope theta");
  if (c->window < 0 || c->global_every < 0) return fail(MEBP_EINVAL, "negative window / global_every");
  if (c->lora_mask >> MEBP_NPROJ) return fail(MEBP_EINVAL, "lora_mask has bits beyond the 7 projections");
  if (c->lora_mask && c->lora_rank != 8 && c->lora_rank != 16)
    return fail(MEBP_EUNSUPPORTED, "lora_rank %d not in {8, 16}", c->lora_rank);
  if (c->lora_mask && !isfinite(c->lora_alpha)) return fail(MEBP_EINVAL, "bad lora_alpha");
  if (c->arch >> 4) return fail(MEBP_EINVAL, "arch has unknown bits 0x%x", c->arch);
  return MEBP_OK;
}

int check_shape(int B, int T) {
  if (B < 1 || T < 1) return fail(MEBP_EINVAL, "B=%d T=%d must be >= 1", B, T);
  if ((long long)B * T > (1LL << 24)) return fail(MEBP_EUNSUPPORTED, "B*T=%lld too large", (long long)B * T);
  return MEBP_OK;
}

int check_ws(const mebp_config* c, int B, int T, void* ws, size_t ws_bytes) {
  const size_t need = mebp_workspace_bytes(c, B, T);
  if (!ws) return fail(MEBP_EINVAL, "workspace is NULL");
  if (!aligned(ws, 256)) return fail(MEBP_EINVAL, "workspace not 256-byte aligned");
  if (ws_bytes < need) return fail(MEBP_EWORKSPACE, "workspace %zu bytes < required %zu", ws_bytes, need);
  return MEBP_OK;
}

int check_q4(const mebp_q4* w, const char* what) {
  if (!w || !w->q4 || !w->scale) return fail(MEBP_EINVAL, "%s: NULL compressed weight", what);
  if (!aligned(w->q4, 4) || !aligned(w->scale, 2)) return fail(MEBP_EINVAL, "%s: misaligned weight", what);
  return MEBP_OK;
}

int check_act(const void* p, const char* what) {
  if (!p) return fail(MEBP_EINVAL, "%s is NULL", what);
  if (!aligned(p, 16)) return fail(MEBP_EINVAL, "%s not 16-byte aligned", what);
  return MEBP_OK;
}

const char* kProjName[MEBP_NPROJ] = {"q", "k", "v", "o", "gate", "up", "down"};

int check_layer(const mebp_config* c, int layer, const mebp_layer_base* base, const mebp_layer_lora* lora) {
  if (layer < 0 || layer >= c->n_layers) return fail(MEBP_EINVAL, "layer %d out of range", layer);
  if (!base) return fail(MEBP_EINVAL, "base is NULL");
  if (!lora) return fail(MEBP_EINVAL, "lora is NULL");
  for (int p = 0; p < MEBP_NPROJ; ++p) {
    int e = check_q4(&base->w[p], kProjName[p]);
    if (e) return e;
    if (c->lora_mask >> p & 1) {
      if (!lora->A[p] || !lora->B[p]) return fail(MEBP_EINVAL, "LoRA %s: NULL A or B", kProjName[p]);
      if (!aligned(lora->A[p], 16) || !aligned(lora->B[p], 16))
        return fail(MEBP_EINVAL, "LoRA %s: A or B not 16-byte aligned", kProjName[p]);
    }
  }
  if (!base->norm_attn || !base->norm_mlp) return fail(MEBP_EINVAL, "NULL norm weight");
  if (!aligned(base->norm_attn, 16) || !aligned(base->norm_mlp, 16))
    return fail(MEBP_EINVAL, "norm weight not 16-byte aligned");
  const float* extra[7] = {base->bias[0], base->bias[1], base->bias[2], base->q_norm, base->k_norm,
                           base->post_attn_norm, base->post_mlp_norm};
  const uint32_t need[7] = {MEBP_ARCH_QKV_BIAS, MEBP_ARCH_QKV_BIAS, MEBP_ARCH_QKV_BIAS, MEBP_ARCH_QK_NORM,
                            MEBP_ARCH_QK_NORM, MEBP_ARCH_SANDWICH, MEBP_ARCH_SANDWICH};
  for (int i = 0; i < 7; ++i)
    if ((c->arch & need[i]) && (!extra[i] || !aligned(extra[i], 16)))
      return fail(MEBP_EINVAL, "layer %d: architecture weight %d NULL or not 16-byte aligned", layer, i);
  return MEBP_OK;
}

int check_grads(const mebp_config* c, const mebp_layer_lora_grad* g) {
  if (!g) return c->lora_mask ? fail(MEBP_EINVAL, "grads is NULL") : MEBP_OK;
  for (int p = 0; p < MEBP_NPROJ; ++p)
    if ((c->lora_mask >> p & 1) && (!g->dA[p] || !g->dB[p]))
      return fail(MEBP_EINVAL, "LoRA grad %s: NULL dA or dB", kProjName[p]);
  return MEBP_OK;
}

// ------------------------------------------------------------------ shapes
struct Dims {
  int N, d, qd, kvd, F, r;
  int in[MEBP_NPROJ], out[MEBP_NPROJ];
  float s;
};
Dims dims(const mebp_config* c, int B, int T) {
  Dims D;
  D.N = B * T;
  D.d = c->hidden;
  D.qd = c->n_heads * c->head_dim;
  D.kvd = c->n_kv_heads * c->head_dim;
  D.F = c->ffn;
  D.r = c->lora_rank;
  D.s = c->lora_mask ? c->lora_alpha / (float)c->lora_rank : 0.f;
  const int in[MEBP_NPROJ] = {D.d, D.d, D.d, D.qd, D.d, D.d, D.F};
  const int out[MEBP_NPROJ] = {D.qd, D.kvd, D.kvd, D.d, D.F, D.F, D.d};
  for (int p = 0; p < MEBP_NPROJ; ++p) {
    D.in[p] = in[p];
    D.out[p] = out[p];
  }
  return D;
}
bool is_global(const mebp_config* c, int l) { return c->global_every == 0 || (l + 1) % c->global_every == 0; }

// ------------------------------------------------------------------ building blocks
struct Ctx {
  const mebp_config* c;
  Dims D;
  int B, T;
  void* ws;
  Layout L;
  hipStream_t st;
  int set;        // copy of the per-layer activation slots (0 or 1)
  int split_set;  // copy of the split-K scratch (0 or 1)
  // When set: the LoRA weight-gradient kernels of the backward run on `aux` after waiting
  // for `ev_lr` (recorded on st); the caller joins aux before the activations they read
  // are rewritten.
  hipStream_t aux;
  hipEvent_t ev_lr;  // recorded on st, waited for by aux
  hipEvent_t ev_du;  // recorded on aux, waited for by st
  bool* aux_used;
};

// The workspace slot `s` as seen by this context (its activation set and scratch copy).
template <class Tp>
Tp* xs(const Ctx& x, int s) {
  const int which = s == S_SPLIT ? x.split_set : x.set;
  return (Tp*)((char*)x.ws + (which ? x.L.off1[s] : x.L.off[s]));
}

SplitScratch split_scratch(const Ctx& x) {
  SplitScratch sc;
  sc.part = xs<float>(x, S_SPLIT);
  sc.part_floats = x.L.split_floats;
  return sc;
}

float* lu(const Ctx& x, int p) { return xs<float>(x, S_LU) + (size_t)p * x.D.N * x.D.r; }
float* ldu(const Ctx& x, int p) { return xs<float>(x, S_LDU) + (size_t)p * x.D.N * x.D.r; }
bool adapted(const Ctx& x, int p) { return (x.c->lora_mask >> p) & 1; }

NtSeg nt_seg(const Ctx& x, const mebp_layer_base* base, const mebp_layer_lora* lora, int p, void* out, int ldo,
             const float* resid, int ldr) {
  NtSeg s{};
  s.q4 = base->w[p].q4;
  s.scale = base->w[p].scale;
  s.N = x.D.out[p];
  s.lora_u = adapted(x, p) ? lu(x, p) : nullptr;
  s.lora_B = adapted(x, p) ? lora->B[p] : nullptr;
  s.out = out;
  s.ldo = ldo;
  s.resid = resid;
  s.ldr = ldr;
  return s;
}

NtArgs nt_args(const Ctx& x, const f16* X, int K, std::initializer_list<NtSeg> segs) {
  NtArgs a{};
  a.X = X;
  a.lda = K;
  a.M = x.D.N;
  a.K = K;
  for (const NtSeg& s : segs) a.seg[a.nseg++] = s;
  a.lora_s = x.D.s;
  a.r = x.D.r;
  const SplitScratch sc = split_scratch(x);
  a.part = sc.part;
  a.part_floats = sc.part_floats;
  a.eps = x.c->rms_eps;
  return a;
}

void set_scratch(const Ctx& x, TnArgs& t) {
  const SplitScratch sc = split_scratch(x);
  t.part = sc.part;
  t.part_floats = sc.part_floats;
  // one copy: the transposed products run on the context's main stream, one after another
  t.w16 = slot<uint16_t>(x.ws, x.L, S_W16);
  t.w16_elems = x.L.w16_elems;
}

TnSeg tn_seg(const Ctx& x, const mebp_layer_base* base, const mebp_layer_lora* lora, int p, const bf16* G) {
  TnSeg s{};
  s.G = G;
  s.ldg = x.D.out[p];
  s.q4 = base->w[p].q4;
  s.scale = base->w[p].scale;
  s.N = x.D.out[p];
  s.lora_du = adapted(x, p) ? ldu(x, p) : nullptr;
  s.lora_A = adapted(x, p) ? lora->A[p] : nullptr;
  return s;
}

// Run `launch` on the context's auxiliary stream once everything enqueued so far on its
// main stream is done (or inline without one); *ready gets the event that marks its end.
template <class F>
hipError_t on_aux(const Ctx& x, hipEvent_t* ready, F&& launch) {
  *ready = nullptr;
  if (!x.aux) return launch(x.st);
  hipError_t e;
  if ((e = hipEventRecord(x.ev_lr, x.st)) != hipSuccess) return e;
  if ((e = hipStreamWaitEvent(x.aux, x.ev_lr, 0)) != hipSuccess) return e;
  if (x.aux_used) *x.aux_used = true;
  if ((e = launch(x.aux)) != hipSuccess) return e;
  if ((e = hipEventRecord(x.ev_du, x.aux)) != hipSuccess) return e;
  *ready = x.ev_du;
  return hipSuccess;
}

// u_p = X A_p^T for the adapted projections among `ps` (LoRA down-projection; X fp16),
// one launch for all of them; the consuming GEMM waits for *ready.
hipError_t lora_down(const Ctx& x, const mebp_layer_lora* lora, const f16* X, int K, std::initializer_list<int> ps,
                     hipEvent_t* ready) {
  *ready = nullptr;
  LoraRowsArgs a{};
  a.M = x.D.N;
  a.r = x.D.r;
  a.wt = 0;
  a.s = 1.0f;
  for (int p : ps) {
    if (!adapted(x, p)) continue;
    a.job[a.njobs++] = LoraRowsJob{X, K, K, lora->A[p], lu(x, p)};
  }
  if (a.njobs == 0) return hipSuccess;
  return on_aux(x, ready, [&](hipStream_t st) { return launch_lora_rows(a, 0, st); });
}

// LoRA backward of the adapted projections among `ps`, with output gradients G_p (bf16
// [N][out_p]) and the shared input X (fp16 [N][in]): du = s G B, dB = s G^T u, dA = du^T X.
// Three launches for all of them. The input-gradient GEMM that adds du A waits for *ready;
// dB and dA feed nothing later in the backward and follow du on the same stream.
hipError_t lora_bwd(const Ctx& x, const mebp_layer_lora* lora, const mebp_layer_lora_grad* grads,
                    std::initializer_list<int> ps, std::initializer_list<const bf16*> Gs, const f16* X,
                    hipEvent_t* ready) {
  *ready = nullptr;
  const Dims& D = x.D;
  LoraRowsArgs ra{};
  ra.M = D.N;
  ra.r = D.r;
  ra.wt = 1;
  ra.s = D.s;
  LoraOuterArgs ob{}, oa{};
  ob.M = oa.M = D.N;
  ob.r = oa.r = D.r;
  ob.layout = 0;
  oa.layout = 1;
  ob.part = oa.part = xs<float>(x, S_PART);
  ob.part_floats = oa.part_floats = x.L.lora_part_floats;
  auto g = Gs.begin();
  for (int p : ps) {
    const bf16* G = *g++;
    if (!adapted(x, p)) continue;
    ra.job[ra.njobs++] = LoraRowsJob{G, D.out[p], D.out[p], lora->B[p], ldu(x, p)};
    ob.job[ob.njobs++] = LoraOuterJob{G, D.out[p], D.out[p], lu(x, p), grads->dB[p], D.s};
    oa.job[oa.njobs++] = LoraOuterJob{X, D.in[p], D.in[p], ldu(x, p), grads->dA[p], 1.0f};
  }
  if (ra.njobs == 0) return hipSuccess;
  hipError_t e = on_aux(x, ready, [&](hipStream_t st) { return launch_lora_rows(ra, 1, st); });
  if (e != hipSuccess) return e;
  hipStream_t so = x.aux ? x.aux : x.st;
  e = launch_lora_outer(ob, 1, so);
  if (e != hipSuccess) return e;
  return launch_lora_outer(oa, 0, so);
}

// Forward of one layer. keep=false: full forward to x_out. keep=true: recompute for the
// backward (stops after z and its LoRA down-projection; x_out unused).
// next_norm (forward loop only): the RMSNorm weights of the next block's input norm; the
// down projection's split-K finalize then also writes that block's normalised input (into
// `next_out`, default the activation slot `a`; one row kernel fewer per layer), and a_ready
// tells the next layer to skip its own input norm.
int layer_forward(const Ctx& x, int l, const mebp_layer_base* base, const mebp_layer_lora* lora, const float* x_in,
                  float* x_out, const float* rope, bool keep, const float* next_norm = nullptr,
                  bool a_ready = false, f16* next_out = nullptr) {
  const mebp_config* c = x.c;
  const Dims& D = x.D;
  f16* a = xs<f16>(x, S_A);
  f16* q = xs<f16>(x, S_Q);
  f16* k = xs<f16>(x, S_K);
  f16* v = xs<f16>(x, S_V);
  f16* o = xs<f16>(x, S_O);
  float* h = xs<float>(x, S_H);
  f16* cc = xs<f16>(x, S_C);
  f16* g = xs<f16>(x, S_G);
  f16* u = xs<f16>(x, S_U);
  f16* z = xs<f16>(x, S_Z);

  if (!a_ready) HIP_TRY(launch_rmsnorm_fwd(x_in, base->norm_attn, D.N, D.d, c->rms_eps, a, nullptr, x.st));
  hipEvent_t lr;
  HIP_TRY(lora_down(x, lora, a, D.d, {MEBP_Q, MEBP_K, MEBP_V}, &lr));
  // bias and per-head norm come between the projection and RoPE: then RoPE moves out of the
  // GEMM's follow-up into the kernel that applies them
  const bool qk_post = c->arch & (MEBP_ARCH_QKV_BIAS | MEBP_ARCH_QK_NORM);
  const bool sandwich = c->arch & MEBP_ARCH_SANDWICH;
  {
    // q, k, v projections with RoPE applied to q and k on the way out
    NtSeg qs = nt_seg(x, base, lora, MEBP_Q, q, D.qd, nullptr, 0), ks = nt_seg(x, base, lora, MEBP_K, k, D.kvd, nullptr, 0);
    qs.rope = ks.rope = qk_post ? 0 : 1;
    NtArgs na = nt_args(x, a, D.d, {qs, ks, nt_seg(x, base, lora, MEBP_V, v, D.kvd, nullptr, 0)});
    na.rope_cs = rope;
    na.rope_T = x.T;
    na.rope_dh = c->head_dim;
    HIP_TRY(launch_gemm_nt(na, NT_STORE_F16, x.st, lr));
  }
  if (qk_post) {
    const bool bias = c->arch & MEBP_ARCH_QKV_BIAS, qkn = c->arch & MEBP_ARCH_QK_NORM;
    HIP_TRY(launch_qkv_post(q, D.qd, D.N, x.T, c->n_heads, c->head_dim, bias ? base->bias[0] : nullptr,
                            qkn ? base->q_norm : nullptr, c->rms_eps, xs<f16>(x, S_QPRE), rope, 1, x.st));
    HIP_TRY(launch_qkv_post(k, D.kvd, D.N, x.T, c->n_kv_heads, c->head_dim, bias ? base->bias[1] : nullptr,
                            qkn ? base->k_norm : nullptr, c->rms_eps, xs<f16>(x, S_KPRE), rope, 1, x.st));
    if (bias)
      HIP_TRY(launch_qkv_post(v, D.kvd, D.N, x.T, c->n_kv_heads, c->head_dim, base->bias[2], nullptr, c->rms_eps,
                              nullptr, rope, 0, x.st));
  }
  AttnArgs at{};
  at.q = q; at.k = k; at.v = v; at.ldq = D.qd; at.ldk = D.kvd;
  at.B = x.B; at.T = x.T; at.Hq = c->n_heads; at.Hkv = c->n_kv_heads; at.dh = c->head_dim;
  at.window = is_global(c, l) ? 0 : c->window;
  at.o = o; at.lse = xs<float>(x, S_LSE);
  HIP_TRY(launch_attn_fwd(at, split_scratch(x), x.st));
  HIP_TRY(lora_down(x, lora, o, D.qd, {MEBP_O}, &lr));
  if (sandwich) {
    // t = o-projection (kept for the backward), h = x + RMSNorm(t), c = RMSNorm(h)
    float* to = xs<float>(x, S_TO);
    HIP_TRY(launch_gemm_nt(nt_args(x, o, D.qd, {nt_seg(x, base, lora, MEBP_O, to, D.d, nullptr, 0)}), NT_STORE_F32, x.st,
                           lr));
    HIP_TRY(launch_resid_rmsnorm(x_in, to, base->post_attn_norm, D.N, D.d, c->rms_eps, h, x.st));
    HIP_TRY(launch_rmsnorm_fwd(h, base->norm_mlp, D.N, D.d, c->rms_eps, cc, nullptr, x.st));
  } else {
    // h = x + o-projection, then c = RMSNorm(h)
    NtArgs na = nt_args(x, o, D.qd, {nt_seg(x, base, lora, MEBP_O, h, D.d, x_in, D.d)});
    na.norm_w = base->norm_mlp;
    na.norm_out = cc;
    HIP_TRY(launch_gemm_nt(na, NT_STORE_F32, x.st, lr));
  }
  HIP_TRY(lora_down(x, lora, cc, D.d, {MEBP_GATE, MEBP_UP}, &lr));
  {
    // g, u projections and z = act(g) * u (g and u kept only for the backward)
    NtArgs na = nt_args(x, cc, D.d, {nt_seg(x, base, lora, MEBP_GATE, g, D.F, nullptr, 0),
                                     nt_seg(x, base, lora, MEBP_UP, u, D.F, nullptr, 0)});
    na.gated = 1;
    na.act = c->act;
    na.z_out = z;
    na.store_gu = keep;
    HIP_TRY(launch_gemm_nt(na, NT_STORE_F16, x.st, lr));
  }
  HIP_TRY(lora_down(x, lora, z, D.F, {MEBP_DOWN}, &lr));
  if (sandwich) {
    // t = down-projection (the backward needs it, so the recompute runs it too), y = h + RMSNorm(t)
    float* td = xs<float>(x, S_TD);
    HIP_TRY(launch_gemm_nt(nt_args(x, z, D.F, {nt_seg(x, base, lora, MEBP_DOWN, td, D.d, nullptr, 0)}), NT_STORE_F32,
                           x.st, lr));
    if (!keep) HIP_TRY(launch_resid_rmsnorm(h, td, base->post_mlp_norm, D.N, D.d, c->rms_eps, x_out, x.st));
  } else if (!keep) {
    NtArgs na = nt_args(x, z, D.F, {nt_seg(x, base, lora, MEBP_DOWN, x_out, D.d, h, D.d)});
    if (next_norm) {
      na.norm_w = next_norm;  // y = h + down(z), and the next block's input RMSNorm(y)
      na.norm_out = next_out ? next_out : a;
    }
    HIP_TRY(launch_gemm_nt(na, NT_STORE_F32, x.st, lr));
  } else if (lr)
    HIP_TRY(hipStreamWaitEvent(x.st, lr, 0));  // u of the down projection is read by the backward
  return MEBP_OK;
}

// dy_bf16_ready: the context's dy_bf16 slot already holds bf16(dy) (written by the
// block above in the same training step). On return the other set's slot holds bf16(dx)
// when dx is computed.
// The backward of one layer from the intermediates of its recomputed forward (already in
// the context's activation set).
int layer_backward_only(const Ctx& x, int l, const mebp_layer_base* base, const mebp_layer_lora* lora,
                        const float* x_ckpt, const float* dy, float* dx, const mebp_layer_lora_grad* grads,
                        const float* rope, bool dy_bf16_ready) {
  const mebp_config* c = x.c;
  const Dims& D = x.D;
  f16* a = xs<f16>(x, S_A);
  f16* q = xs<f16>(x, S_Q);
  f16* k = xs<f16>(x, S_K);
  f16* v = xs<f16>(x, S_V);
  f16* o = xs<f16>(x, S_O);
  float* h = xs<float>(x, S_H);
  f16* cc = xs<f16>(x, S_C);
  f16* g = xs<f16>(x, S_G);
  f16* u = xs<f16>(x, S_U);
  f16* z = xs<f16>(x, S_Z);
  bf16* dyb = xs<bf16>(x, S_DYB);
  Ctx other = x;
  other.set ^= 1;
  bf16* dxb = xs<bf16>(other, S_DYB);  // bf16(dx) for the layer below
  float* dc = xs<float>(x, S_DC);
  float* dh = xs<float>(x, S_DH);
  bf16* dhb = xs<bf16>(x, S_DHB);
  bf16* dO = xs<bf16>(x, S_DO);
  bf16* dq = xs<bf16>(x, S_DQ);
  bf16* dk = xs<bf16>(x, S_DK);
  bf16* dv = xs<bf16>(x, S_DV);
  float* da = xs<float>(x, S_DA);

  const bool sandwich = c->arch & MEBP_ARCH_SANDWICH;
  // y = h + down(z)   (sandwich: y = h + RMSNorm(t), t = down(z): the down projection's
  // gradient is the norm's backward of dy)
  bf16* gdown = dyb;
  if (sandwich) {
    gdown = xs<bf16>(x, S_DTB);
    HIP_TRY(launch_rmsnorm_bwd(xs<float>(x, S_TD), base->post_mlp_norm, dy, nullptr, D.N, D.d, c->rms_eps, nullptr,
                               gdown, x.st));
  } else if (!dy_bf16_ready) {
    HIP_TRY(launch_f32_to_bf16(dy, dyb, (size_t)D.N * D.d, x.st));
  }
  hipEvent_t lr;
  HIP_TRY(lora_bwd(x, lora, grads, {MEBP_DOWN}, {gdown}, z, &lr));
  {
    TnArgs t{};
    set_scratch(x, t);
    t.M = D.N; t.Kout = D.F; t.nseg = 1; t.r = D.r;
    t.seg[0] = tn_seg(x, base, lora, MEBP_DOWN, gdown);
    t.g = g; t.u = u; t.ldgu = D.F; t.act = c->act;
    HIP_TRY(launch_gemm_tn(t, TN_ACT_BWD, TN_A_BF16, x.st, lr));  // g <- dg, u <- d(up)
  }
  // z = act(gate(c)) * up(c)
  bf16* dg = (bf16*)g;  // the act-backward epilogue left bf16 dg / du in the g / u buffers
  bf16* dup = (bf16*)u;
  HIP_TRY(lora_bwd(x, lora, grads, {MEBP_GATE, MEBP_UP}, {dg, dup}, cc, &lr));
  {
    TnArgs t{};
    set_scratch(x, t);
    t.M = D.N; t.Kout = D.d; t.nseg = 2; t.r = D.r;
    t.seg[0] = tn_seg(x, base, lora, MEBP_GATE, dg);
    t.seg[1] = tn_seg(x, base, lora, MEBP_UP, dup);
    t.out = dc; t.ldo = D.d;
    // c = RMSNorm(h): dh = dy + rmsnorm_bwd(h, dc)
    t.norm_x = h; t.norm_w = base->norm_mlp; t.resid2 = dy; t.out2 = dh; t.out2b = dhb; t.eps = c->rms_eps;
    HIP_TRY(launch_gemm_tn(t, TN_STORE_F32, TN_A_BF16, x.st, lr));
  }
  // h = x + o(O)   (sandwich: h = x + RMSNorm(t), t = o(O))
  bf16* go = dhb;
  if (sandwich) {
    go = xs<bf16>(x, S_DTOB);
    HIP_TRY(launch_rmsnorm_bwd(xs<float>(x, S_TO), base->post_attn_norm, dh, nullptr, D.N, D.d, c->rms_eps, nullptr,
                               go, x.st));
  }
  HIP_TRY(lora_bwd(x, lora, grads, {MEBP_O}, {go}, o, &lr));
  {
    TnArgs t{};
    set_scratch(x, t);
    t.M = D.N; t.Kout = D.qd; t.nseg = 1; t.r = D.r;
    t.seg[0] = tn_seg(x, base, lora, MEBP_O, go);
    t.outb = dO; t.ldo = D.qd;
    // the attention backward's delta = rowsum(dO * O) comes with dO
    t.delta_o = o; t.delta = xs<float>(x, S_DELTA); t.delta_T = x.T; t.delta_dh = c->head_dim;
    HIP_TRY(launch_gemm_tn(t, TN_STORE_BF16, TN_A_BF16, x.st, lr));
  }
  // attention (RoPE backward fused into the dq / dk stores)
  {
    AttnArgs at{};
    at.q = q; at.k = k; at.v = v; at.ldq = D.qd; at.ldk = D.kvd;
    at.B = x.B; at.T = x.T; at.Hq = c->n_heads; at.Hkv = c->n_kv_heads; at.dh = c->head_dim;
    at.window = is_global(c, l) ? 0 : c->window;
    at.o = o; at.lse = xs<float>(x, S_LSE);
    at.dO = dO; at.cs = rope; at.dq = dq; at.dk = dk; at.dv = dv;
    if (x.aux && x.aux_used) *x.aux_used = true;
    HIP_TRY(launch_attn_bwd(at, xs<float>(x, S_DELTA), split_scratch(x), x.st, x.aux, x.ev_lr, x.ev_du, true));
  }
  if (c->arch & MEBP_ARCH_QK_NORM) {
    // through the per-head norms (the biases are frozen and need no gradient)
    HIP_TRY(launch_headnorm_bwd(xs<f16>(x, S_QPRE), D.qd, D.N, c->n_heads, c->head_dim, base->q_norm, c->rms_eps, dq,
                                D.qd, x.st));
    HIP_TRY(launch_headnorm_bwd(xs<f16>(x, S_KPRE), D.kvd, D.N, c->n_kv_heads, c->head_dim, base->k_norm, c->rms_eps,
                                dk, D.kvd, x.st));
  }
  HIP_TRY(lora_bwd(x, lora, grads, {MEBP_Q, MEBP_K, MEBP_V}, {dq, dk, dv}, a, &lr));
  if (dx) {
    TnArgs t{};
    set_scratch(x, t);
    t.M = D.N; t.Kout = D.d; t.nseg = 3; t.r = D.r;
    t.seg[0] = tn_seg(x, base, lora, MEBP_Q, dq);
    t.seg[1] = tn_seg(x, base, lora, MEBP_K, dk);
    t.seg[2] = tn_seg(x, base, lora, MEBP_V, dv);
    t.out = da; t.ldo = D.d;
    // a = RMSNorm(x): dx = dh + rmsnorm_bwd(x, da)  (dx may alias dy: dy is no longer read)
    t.norm_x = x_ckpt; t.norm_w = base->norm_attn; t.resid2 = dh; t.out2 = dx; t.out2b = dxb; t.eps = c->rms_eps;
    HIP_TRY(launch_gemm_tn(t, TN_STORE_F32, TN_A_BF16, x.st, lr));
  }
  return MEBP_OK;
}

// Recompute (Algorithm 1's second loop: forward from the checkpoint) then backward.
int layer_backward(const Ctx& x, int l, const mebp_layer_base* base, const mebp_layer_lora* lora,
                   const float* x_ckpt, const float* dy, float* dx, const mebp_layer_lora_grad* grads,
                   const float* rope, bool dy_bf16_ready = false) {
  const int e = layer_forward(x, l, base, lora, x_ckpt, nullptr, rope, true);
  if (e) return e;
  return layer_backward_only(x, l, base, lora, x_ckpt, dy, dx, grads, rope, dy_bf16_ready);
}

// The final block (Sec. 4.2: the final linear layer and the loss layer are one block of the
// checkpointed graph): final RMSNorm, logits against the tied int4 embedding, next-token
// cross-entropy and its gradient. The vocabulary is processed in chunks so that only one
// chunk's logits exist at a time: per chunk the logits product (tile statistics and
// tile-relative fp16 logits), the merge of its statistics into each row's running maximum
// and sum, its softmax weights relative to the running maximum (in place, bf16), and the dH
// product accumulated into an fp32 row accumulator rescaled to the new maximum. Every logit
// is computed once (4 N d V flops for both products).
int lm_head(const Ctx& x, const mebp_q4* emb, const float* norm_final, const float* x_last, const int32_t* ids,
            float* loss, float* dx_last, bf16* dx_last_bf16, bool hf_ready = false) {
  const mebp_config* c = x.c;
  const Dims& D = x.D;
  const int V = c->vocab, d = D.d, N = D.N;
  int32_t* tgt = xs<int32_t>(x, S_TGT);
  f16* hf = xs<f16>(x, S_HF);
  _Float16* logits = xs<_Float16>(x, S_LOGITS);
  float2* stats = xs<float2>(x, S_STATS);
  float* lse = xs<float>(x, S_LSEV);
  float* tl = xs<float>(x, S_TGTLOGIT);
  float* rl = xs<float>(x, S_ROWLOSS);
  float* dhf = xs<float>(x, S_DHF);
  float* part = xs<float>(x, S_LMPART);
  float* mrun = xs<float>(x, S_CEMAX);
  float* lrun = xs<float>(x, S_CESUM);
  float* alpha = xs<float>(x, S_CEALPHA);
  const float inv_n = 1.0f / (float)((long long)x.B * (x.T - 1));
  const int Vc = x.L.lm_chunk, ldt = x.L.ntiles, kg = (d + 31) / 32;

  HIP_TRY(launch_targets(ids, x.B, x.T, c->vocab, tgt, x.st));
  if (!hf_ready) HIP_TRY(launch_rmsnorm_fwd(x_last, norm_final, N, d, c->rms_eps, hf, nullptr, x.st));
  for (int v0 = 0; v0 < V; v0 += Vc) {
    const int w = V - v0 < Vc ? V - v0 : Vc;
    const int first = v0 == 0;
    const uint8_t* eq4 = emb->q4 + (size_t)v0 * (d / 2);
    const uint16_t* esc = emb->scale + (size_t)v0 * kg;
    {
      NtArgs a{};
      a.X = hf; a.lda = d; a.M = N; a.K = d; a.nseg = 1;
      a.seg[0].q4 = eq4; a.seg[0].scale = esc; a.seg[0].N = w; a.seg[0].tile0 = 0;
      a.seg[0].out = logits; a.seg[0].ldo = Vc;
      a.stats = stats; a.tgt = tgt; a.tgt_logit = tl; a.ntiles = ldt; a.vbase = v0;
      HIP_TRY(launch_gemm_nt(a, NT_LOGITS, x.st));
    }
    HIP_TRY(launch_ce_chunk_stats(stats, ldt, gemm_logit_stat_tiles(w), N, mrun, lrun, alpha, first, x.st));
    HIP_TRY(launch_ce_probs(reinterpret_cast<uint16_t*>(logits), N, w, Vc, stats, ldt, mrun, tgt, v0, x.st));
    {
      TnArgs t{};
      t.M = N; t.Kout = d; t.nseg = 1; t.r = 0;
      t.seg[0].G = (const bf16*)logits; t.seg[0].ldg = Vc;
      t.seg[0].q4 = eq4; t.seg[0].scale = esc; t.seg[0].N = w;
      t.out = part; t.ldo = d; t.splits = lm_head_splits(N, d, w);
      t.w16 = slot<uint16_t>(x.ws, x.L, S_W16); t.w16_elems = x.L.w16_elems;
      HIP_TRY(launch_gemm_tn(t, TN_PARTIAL_F32, TN_A_BF16, x.st));
      HIP_TRY(launch_ce_dh_accum(part, t.splits, N, d, alpha, first, dhf, x.st));
    }
  }
  HIP_TRY(launch_ce_final(N, d, emb->q4, emb->scale, tgt, tl, mrun, lrun, inv_n, dhf, lse, rl, x.st));
  HIP_TRY(launch_ce_loss(rl, tgt, N, inv_n, loss, x.st));
  HIP_TRY(launch_rmsnorm_bwd(x_last, norm_final, dhf, nullptr, N, d, c->rms_eps, dx_last, dx_last_bf16, x.st));
  return MEBP_OK;
}

Ctx make_ctx(const mebp_config* c, int B, int T, void* ws, mebp_stream_t stream) {
  Ctx x;
  x.c = c;
  x.D = dims(c, B, T);
  x.B = B;
  x.T = T;
  x.ws = ws;
  make_layout(c, B, T, &x.L);
  x.st = (hipStream_t)stream;
  x.set = 0;
  x.split_set = 0;
  x.aux = nullptr;
  x.ev_lr = nullptr;
  x.ev_du = nullptr;
  x.aux_used = nullptr;
  return x;
}

int rope_table(const Ctx& x, int l, float** out) {
  const bool glob = is_global(x.c, l);
  float* cs = xs<float>(x, glob ? S_ROPE_G : S_ROPE_L);
  HIP_TRY(launch_rope_table(x.T, x.c->head_dim, glob ? x.c->rope_theta_global : x.c->rope_theta_local, cs, x.st));
  *out = cs;
  return MEBP_OK;
}

// ------------------------------------------------------------------ side stream
// The training step runs the recompute of layer l-1 on a second stream of the caller's
// device while layer l is backpropagated on the caller's stream, and the LoRA dA / dB
// kernels on a third. The streams and their events are created on the first step on a
// device outside of stream capture (a step captured before that runs on the caller's
// stream alone). Enqueueing a step holds the
// device's lock, so concurrent host threads do not interleave on the shared events.
struct SideStream {
  hipStream_t st = nullptr, aux = nullptr;
  hipEvent_t ev_fwd = nullptr, ev_rec = nullptr, ev_bwd = nullptr, ev_lr = nullptr, ev_aux = nullptr;
  hipEvent_t ev_du = nullptr;
  std::mutex mu;
};

SideStream* side_stream(hipStream_t main) {
  static std::mutex map_mu;
  static std::map<int, SideStream*> by_dev;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return nullptr;
  std::lock_guard<std::mutex> g(map_mu);
  auto it = by_dev.find(dev);
  if (it != by_dev.end()) return it->second;
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(main, &cs) != hipSuccess || cs != hipStreamCaptureStatusNone) return nullptr;
  SideStream* s = new SideStream();
  if (hipStreamCreateWithFlags(&s->st, hipStreamNonBlocking) != hipSuccess ||
      hipStreamCreateWithFlags(&s->aux, hipStreamNonBlocking) != hipSuccess ||
      hipEventCreateWithFlags(&s->ev_lr, hipEventDisableTiming) != hipSuccess ||
      hipEventCreateWithFlags(&s->ev_aux, hipEventDisableTiming) != hipSuccess ||
      hipEventCreateWithFlags(&s->ev_du, hipEventDisableTiming) != hipSuccess ||
      hipEventCreateWithFlags(&s->ev_fwd, hipEventDisableTiming) != hipSuccess ||
      hipEventCreateWithFlags(&s->ev_rec, hipEventDisableTiming) != hipSuccess ||
      hipEventCreateWithFlags(&s->ev_bwd, hipEventDisableTiming) != hipSuccess) {
    (void)hipGetLastError();
    return nullptr;  // (leaks the partial set; the step then runs on one stream)
  }
  by_dev[dev] = s;
  return s;
}

// Checkpoint offload (the memory-mapped checkpoints of Sec. 3, "Runtime implementation"):
// x_i lives in device ring slot i % R while it is computed and used; a copy stream moves
// every checkpoint to pinned host memory as soon as it is written and brings it back into
// its slot before the reverse loop recomputes that layer. Without it, ring = the caller's
// full checkpoint array (slot i = x_i) and nothing is copied.
struct Offload {
  float* host = nullptr;      // [(L+1)][N][d] pinned host memory
  float* host_dev = nullptr;  // the same memory's device address (null: copies through hipMemcpyAsync)
  int R = 0;              // ring slots
  hipStream_t cp = nullptr;
  hipEvent_t ev_in[MEBP_RING_MAX], ev_out[MEBP_RING_MAX];
  hipEvent_t ev_go = nullptr;
};

struct OffloadStreams {
  hipStream_t cp = nullptr;
  hipEvent_t ev_in[MEBP_RING_MAX], ev_out[MEBP_RING_MAX], ev_go = nullptr;
  bool ok = false;
};

OffloadStreams* offload_streams() {
  static std::mutex mu;
  static std::map<int, OffloadStreams*> by_dev;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return nullptr;
  std::lock_guard<std::mutex> g(mu);
  auto it = by_dev.find(dev);
  if (it != by_dev.end()) return it->second;
  OffloadStreams* o = new OffloadStreams();
  bool ok = hipStreamCreateWithFlags(&o->cp, hipStreamNonBlocking) == hipSuccess &&
            hipEventCreateWithFlags(&o->ev_go, hipEventDisableTiming) == hipSuccess;
  for (int i = 0; ok && i < MEBP_RING_MAX; ++i)
    ok = hipEventCreateWithFlags(&o->ev_in[i], hipEventDisableTiming) == hipSuccess &&
         hipEventCreateWithFlags(&o->ev_out[i], hipEventDisableTiming) == hipSuccess;
  if (!ok) {
    (void)hipGetLastError();
    return nullptr;
  }
  o->ok = true;
  by_dev[dev] = o;
  return o;
}

int train_step_impl(const mebp_config* cfg, const mebp_q4* emb, const mebp_layer_base* layers,
                    const float* norm_final, const mebp_layer_lora* lora, const int32_t* ids, int32_t B, int32_t T,
                    float* ring, Offload* off, float* loss, const mebp_layer_lora_grad* grads, float* dx0, void* ws,
                    mebp_stream_t stream) {
  int e;
  Ctx x = make_ctx(cfg, B, T, ws, stream);
  const size_t stride = (size_t)x.D.N * x.D.d, bytes = stride * sizeof(float);
  const int L = cfg->n_layers;
  auto ck = [&](int i) { return ring + (off ? (size_t)(i % off->R) : (size_t)i) * stride; };
  // x_i still in the ring after the forward loop (the last R checkpoints)
  auto resident = [&](int i) { return !off || i > L - off->R; };
  // D2H of checkpoint i once `after` (a stream that wrote it) has reached this point
  auto save = [&](int i, hipStream_t after) -> int {
    HIP_TRY(hipEventRecord(off->ev_go, after));
    HIP_TRY(hipStreamWaitEvent(off->cp, off->ev_go, 0));
    // (the runtime's device-to-host copy is a kernel that holds many compute units for the
    // whole transfer over the host link; the few-workgroup copy leaves them to the layers)
    if (off->host_dev)
      HIP_TRY(launch_copy_host(ck(i), off->host_dev + (size_t)i * stride, bytes, off->cp));
    else
      HIP_TRY(hipMemcpyAsync(off->host + (size_t)i * stride, ck(i), bytes, hipMemcpyDeviceToHost, off->cp));
    HIP_TRY(hipEventRecord(off->ev_out[i % off->R], off->cp));
    return MEBP_OK;
  };
  // H2D of checkpoint i into its slot once `after` is done with the slot's previous content
  auto fetch = [&](int i, hipStream_t after) -> int {
    HIP_TRY(hipEventRecord(off->ev_go, after));
    HIP_TRY(hipStreamWaitEvent(off->cp, off->ev_go, 0));
    if (off->host_dev)
      HIP_TRY(launch_copy_host(off->host_dev + (size_t)i * stride, ck(i), bytes, off->cp));
    else
      HIP_TRY(hipMemcpyAsync(ck(i), off->host + (size_t)i * stride, bytes, hipMemcpyHostToDevice, off->cp));
    HIP_TRY(hipEventRecord(off->ev_in[i % off->R], off->cp));
    return MEBP_OK;
  };
  float* rope_g = slot<float>(ws, x.L, S_ROPE_G);
  float* rope_l = slot<float>(ws, x.L, S_ROPE_L);
  HIP_TRY(launch_rope_table(T, cfg->head_dim, cfg->rope_theta_global, rope_g, x.st));
  HIP_TRY(launch_rope_table(T, cfg->head_dim, cfg->rope_theta_local, rope_l, x.st));
  const float emb_mul = (cfg->arch & MEBP_ARCH_EMBED_SCALE) ? sqrtf((float)cfg->hidden) : 1.0f;
  HIP_TRY(launch_embed(emb->q4, emb->scale, cfg->hidden, cfg->group, ids, x.D.N, cfg->vocab, ck(0), x.st, emb_mul));
  if (off && (e = save(0, x.st))) return e;
  SideStream* side = side_stream(x.st);
  std::unique_lock<std::mutex> lock;
  if (side) lock = std::unique_lock<std::mutex>(side->mu);
  // forward loop: ckpt[l+1] = forward_l(ckpt[l]); the LoRA down-projections run on the
  // auxiliary stream beside the base GEMMs whose finalize adds them
  {
    Ctx xf = x;
    if (side) {
      xf.aux = side->aux;
      xf.ev_lr = side->ev_lr;
      xf.ev_du = side->ev_du;
    }
    for (int l = 0; l < L; ++l) {
      const float* rope = is_global(cfg, l) ? rope_g : rope_l;
      // the slot of x_{l+1} last held x_{l+1-R}: its copy to the host must be done
      if (off && l + 1 >= off->R) HIP_TRY(hipStreamWaitEvent(x.st, off->ev_out[(l + 1) % off->R], 0));
      // the next layer's input norm rides on this layer's down-projection finalize (not with
      // sandwich norms, whose output norm is a kernel of its own)
      const bool fuse = !(cfg->arch & MEBP_ARCH_SANDWICH);
      const float* nn = !fuse ? nullptr : l + 1 < L ? layers[l + 1].norm_attn : norm_final;
      f16* nout = l + 1 < L ? nullptr : slot<f16>(ws, x.L, S_HF);
      if ((e = layer_forward(xf, l, &layers[l], &lora[l], ck(l), ck(l + 1), rope, false, nn, fuse && l > 0, nout)))
        return e;
      if (off && (e = save(l + 1, x.st))) return e;
    }
  }
  float* g = slot<float>(ws, x.L, S_GRAD);
  const bool hf_fused = !(cfg->arch & MEBP_ARCH_SANDWICH);  // the LM head's input norm ran with the last layer
  // reverse loop: recompute layer l from ckpt[l], backpropagate the upstream gradient
  Ctx top = x;
  top.set = (L - 1) & 1;  // layer l reads bf16(dy) from set l & 1
  bf16* dyb_top = xs<bf16>(top, S_DYB);
  // checkpoints that left the ring come back R layers ahead: x_i returns into its slot
  // after the backward of layer i + R (the slot's previous user), well before layer i's
  // recompute
  // after layer l's backward its slot is free for x_{l-R}; x_{L-R} goes into the slot of
  // x_L, which only the LM head reads, right after the LM head
  auto after_backward = [&](int l, hipStream_t st) -> int {
    if (off && l - off->R >= 0) return fetch(l - off->R, st);
    return MEBP_OK;
  };
  if (!side) {
    // final linear + loss block, then the layers in reverse on the caller's stream
    if ((e = lm_head(x, emb, norm_final, ck(L), ids, loss, g, dyb_top, hf_fused))) return e;
    if (off && L - off->R >= 0 && (e = fetch(L - off->R, x.st))) return e;
    for (int l = L - 1; l >= 0; --l) {
      Ctx b = x;
      b.set = l & 1;
      const float* rope = is_global(cfg, l) ? rope_g : rope_l;
      float* dxl = l > 0 ? g : dx0;
      if (!resident(l)) HIP_TRY(hipStreamWaitEvent(x.st, off->ev_in[l % off->R], 0));
      if ((e = layer_backward(b, l, &layers[l], &lora[l], ck(l), g, dxl, grads ? &grads[l] : nullptr, rope, true)))
        return e;
      if ((e = after_backward(l, x.st))) return e;
    }
  } else {
    // Two streams: the recompute of layer l writes activation set l & 1 on the side stream
    // (with its own split-K scratch) and may start as soon as the backward of layer l + 2,
    // the previous user of that set, is done; the backward of layer l waits for it. The
    // side stream's first wait is on the end of the forward loop (the checkpoints and the
    // LM head's inputs), its last record is waited for by the caller's stream.
    Ctx r = x;
    r.st = side->st;
    r.split_set = 1;
    auto recompute = [&](int l) -> int {
      r.set = l & 1;
      const float* rope = is_global(cfg, l) ? rope_g : rope_l;
      if (!resident(l)) HIP_TRY(hipStreamWaitEvent(side->st, off->ev_in[l % off->R], 0));
      return layer_forward(r, l, &layers[l], &lora[l], ck(l), nullptr, rope, true);
    };
    HIP_TRY(hipEventRecord(side->ev_fwd, x.st));
    HIP_TRY(hipStreamWaitEvent(side->st, side->ev_fwd, 0));
    // (the LM head below is enqueued after this point on the caller's stream and overlaps
    // the first recompute)
    if ((e = recompute(L - 1))) return e;
    HIP_TRY(hipEventRecord(side->ev_rec, side->st));
    if ((e = lm_head(x, emb, norm_final, ck(L), ids, loss, g, dyb_top, hf_fused))) return e;
    if (off && L - off->R >= 0 && (e = fetch(L - off->R, x.st))) return e;
    for (int l = L - 1; l >= 0; --l) {
      HIP_TRY(hipStreamWaitEvent(x.st, side->ev_rec, 0));  // recompute(l) done
      if (l >= 1) {
        // set (l - 1) & 1 was last read by the backward of layer l + 1 (or the forward loop)
        if (l + 1 < L) HIP_TRY(hipStreamWaitEvent(side->st, side->ev_bwd, 0));
        if ((e = recompute(l - 1))) return e;
        HIP_TRY(hipEventRecord(side->ev_rec, side->st));
      }
      Ctx b = x;
      b.set = l & 1;
      bool aux_used = false;
      b.aux = side->aux;
      b.ev_lr = side->ev_lr;
      b.ev_du = side->ev_du;
      b.aux_used = &aux_used;
      const float* rope = is_global(cfg, l) ? rope_g : rope_l;
      float* dxl = l > 0 ? g : dx0;
      if ((e = layer_backward_only(b, l, &layers[l], &lora[l], ck(l), g, dxl, grads ? &grads[l] : nullptr, rope,
                                   true)))
        return e;
      if (aux_used) {
        // the dA / dB kernels of this layer read set l & 1, its bf16(dy) and the shared
        // gradient slots: join them before the next layer's backward or recompute
        HIP_TRY(hipEventRecord(side->ev_aux, side->aux));
        HIP_TRY(hipStreamWaitEvent(x.st, side->ev_aux, 0));
      }
      HIP_TRY(hipEventRecord(side->ev_bwd, x.st));
      if ((e = after_backward(l, x.st))) return e;
    }
  }
  if (off) {
    // every copy of the step is joined into the caller's stream
    HIP_TRY(hipEventRecord(off->ev_go, off->cp));
    HIP_TRY(hipStreamWaitEvent(x.st, off->ev_go, 0));
  }
  return MEBP_OK;
}

}  // namespace

// ==================================================================== public entry points
extern "C" {

size_t mebp_workspace_bytes(const mebp_config* cfg, int32_t B, int32_t T) {
  std::string saved = g_last_error;
  if (check_config(cfg) || check_shape(B, T)) {
    g_last_error = saved;
    return 0;
  }
  Layout L;
  make_layout(cfg, B, T, &L);
  return L.total;
}

size_t mebp_workspace_offset(const mebp_config* cfg, int32_t B, int32_t T, int32_t s) {
  if (s < 0 || s >= S_COUNT || check_config(cfg) || check_shape(B, T)) return (size_t)-1;
  Layout L;
  make_layout(cfg, B, T, &L);
  return L.off[s];
}

const char* mebp_workspace_slot_name(int32_t s) { return (s >= 0 && s < S_COUNT) ? kSlotNames[s] : nullptr; }

const char* mebp_last_error(void) { return g_last_error.c_str(); }

int mebp_set_workspace_guards(int32_t on) { return g_guards.exchange(on ? 1 : 0); }

int mebp_workspace_guard_check(const mebp_config* cfg, int32_t B, int32_t T, void* ws, size_t ws_bytes,
                               mebp_stream_t stream) {
  int e;
  if (!g_guards.load()) return fail(MEBP_EINVAL, "workspace guards are off");
  if ((e = check_config(cfg)) || (e = check_shape(B, T)) || (e = check_ws(cfg, B, T, ws, ws_bytes))) return e;
  Layout L;
  make_layout(cfg, B, T, &L);
  return guard_verdict(L, ws, (hipStream_t)stream);
}

int mebp_layer_forward_ckpt(const mebp_config* cfg, int32_t layer, const mebp_layer_base* base,
                            const mebp_layer_lora* lora, const float* x_in, float* x_out, int32_t B, int32_t T,
                            void* ws, size_t ws_bytes, mebp_stream_t stream) {
  int e;
  if ((e = check_config(cfg)) || (e = check_shape(B, T)) || (e = check_layer(cfg, layer, base, lora)) ||
      (e = check_act(x_in, "x_in")) || (e = check_act(x_out, "x_out")) || (e = check_ws(cfg, B, T, ws, ws_bytes)))
    return e;
  if (x_in == x_out) return fail(MEBP_EINVAL, "x_out must not alias x_in");
  return guarded(cfg, B, T, ws, stream, [&] {
    Ctx x = make_ctx(cfg, B, T, ws, stream);
    float* rope;
    int e2;
    if ((e2 = rope_table(x, layer, &rope))) return e2;
    return layer_forward(x, layer, base, lora, x_in, x_out, rope, false);
  });
}

int mebp_layer_recompute_backward(const mebp_config* cfg, int32_t layer, const mebp_layer_base* base,
                                  const mebp_layer_lora* lora, const float* x_ckpt, const float* dy, float* dx,
                                  const mebp_layer_lora_grad* grads, int32_t B, int32_t T, void* ws, size_t ws_bytes,
                                  mebp_stream_t stream) {
  int e;
  if ((e = check_config(cfg)) || (e = check_shape(B, T)) || (e = check_layer(cfg, layer, base, lora)) ||
      (e = check_act(x_ckpt, "x_ckpt")) || (e = check_act(dy, "dy")) || (e = check_grads(cfg, grads)) ||
      (e = check_ws(cfg, B, T, ws, ws_bytes)))
    return e;
  if (dx && !aligned(dx, 16)) return fail(MEBP_EINVAL, "dx not 16-byte aligned");
  if (dx && dx == x_ckpt) return fail(MEBP_EINVAL, "dx must not alias x_ckpt");
  return guarded(cfg, B, T, ws, stream, [&] {
    Ctx x = make_ctx(cfg, B, T, ws, stream);
    float* rope;
    int e2;
    if ((e2 = rope_table(x, layer, &rope))) return e2;
    return layer_backward(x, layer, base, lora, x_ckpt, dy, dx, grads, rope);
  });
}

}  // extern "C"

namespace {
// Device address of the current device's copy of `scratch`, looked up once per device (with
// that device current) and kept; null on failure (the message is recorded).
void* static_scratch() {
  static std::mutex mu;
  static std::map<int, void*> by_dev;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) {
    fail(MEBP_EHIP, "hipGetDevice: %s", hipGetErrorString(e));
    return nullptr;
  }
  std::lock_guard<std::mutex> g(mu);
  auto it = by_dev.find(dev);
  if (it != by_dev.end()) return it->second;
  void* p = nullptr;
  e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
  if (e != hipSuccess || !p) {
    fail(MEBP_EHIP, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
    return nullptr;
  }
  by_dev[dev] = p;
  return p;
}
}  // namespace

extern "C" {

int mebp_layer_recompute_backward_static(const mebp_config* cfg, int32_t layer, const mebp_layer_base* base,
                                         const mebp_layer_lora* lora, const float* x_ckpt, const float* dy, float* dx,
                                         const mebp_layer_lora_grad* grads, int32_t B, int32_t T,
                                         mebp_stream_t stream) {
  int e;
  if ((e = check_config(cfg)) || (e = check_shape(B, T)) || (e = check_layer(cfg, layer, base, lora)) ||
      (e = check_act(x_ckpt, "x_ckpt")) || (e = check_act(dy, "dy")) || (e = check_grads(cfg, grads)))
    return e;
  if (dx && !aligned(dx, 16)) return fail(MEBP_EINVAL, "dx not 16-byte aligned");
  if (dx && dx == x_ckpt) return fail(MEBP_EINVAL, "dx must not alias x_ckpt");
  // the layer's own slots only: the LM head's are not part of this call
  mebp_config c0 = *cfg;
  c0.vocab = 0;
  const size_t need = mebp_workspace_bytes(&c0, B, T);
  if (need > MEBP_STATIC_SCRATCH_BYTES)
    return fail(MEBP_EWORKSPACE, "layer needs %zu bytes of scratch, more than the %zu the library holds", need,
                (size_t)MEBP_STATIC_SCRATCH_BYTES);
  void* ws = static_scratch();
  if (!ws) return MEBP_EHIP;
  return guarded(&c0, B, T, ws, stream, [&] {
    Ctx x = make_ctx(&c0, B, T, ws, stream);
    float* rope;
    int e2;
    if ((e2 = rope_table(x, layer, &rope))) return e2;
    return layer_backward(x, layer, base, lora, x_ckpt, dy, dx, grads, rope);
  });
}

int mebp_lm_head_ce_backward(const mebp_config* cfg, const mebp_q4* emb, const float* norm_final,
                             const float* x_last, const int32_t* ids, int32_t B, int32_t T, float* loss,
                             float* dx_last, void* ws, size_t ws_bytes, mebp_stream_t stream) {
  int e;
  if ((e = check_config(cfg)) || (e = check_shape(B, T))) return e;
  if (cfg->vocab <= 0) return fail(MEBP_EINVAL, "vocab must be > 0 for the LM head");
  if (T < 2) return fail(MEBP_EINVAL, "T must be >= 2 (no next-token target otherwise)");
  if ((e = check_q4(emb, "embedding")) || (e = check_act(norm_final, "norm_final")) ||
      (e = check_act(x_last, "x_last")) || (e = check_act(dx_last, "dx_last")) || (e = check_ws(cfg, B, T, ws, ws_bytes)))
    return e;
  if (!ids || !aligned(ids, 4)) return fail(MEBP_EINVAL, "ids NULL or misaligned");
  if (!loss || !aligned(loss, 4)) return fail(MEBP_EINVAL, "loss NULL or misaligned");
  return guarded(cfg, B, T, ws, stream, [&] {
    Ctx x = make_ctx(cfg, B, T, ws, stream);
    return lm_head(x, emb, norm_final, x_last, ids, loss, dx_last, xs<bf16>(x, S_DYB));
  });
}

int mebp_embed(const mebp_config* cfg, const mebp_q4* emb, const int32_t* ids, int32_t B, int32_t T, float* x0,
               mebp_stream_t stream) {
  int e;
  if ((e = check_config(cfg)) || (e = check_shape(B, T))) return e;
  if (cfg->vocab <= 0) return fail(MEBP_EINVAL, "vocab must be > 0 for the embedding");
  if ((e = check_q4(emb, "embedding")) || (e = check_act(x0, "x0"))) return e;
  if (!ids || !aligned(ids, 4)) return fail(MEBP_EINVAL, "ids NULL or misaligned");
  const float emb_mul = (cfg->arch & MEBP_ARCH_EMBED_SCALE) ? sqrtf((float)cfg->hidden) : 1.0f;
  HIP_TRY(launch_embed(emb->q4, emb->scale, cfg->hidden, cfg->group, ids, B * T, cfg->vocab, x0, (hipStream_t)stream,
                       emb_mul));
  return MEBP_OK;
}

int check_train_args(const mebp_config* cfg, const mebp_q4* emb, const mebp_layer_base* layers,
                     const float* norm_final, const mebp_layer_lora* lora, const int32_t* ids, int32_t B, int32_t T,
                     float* loss, const mebp_layer_lora_grad* grads, float* dx0, void* ws, size_t ws_bytes) {
  int e;
  if ((e = check_config(cfg)) || (e = check_shape(B, T))) return e;
  if (cfg->vocab <= 0) return fail(MEBP_EINVAL, "vocab must be > 0 for a training step");
  if (T < 2) return fail(MEBP_EINVAL, "T must be >= 2 (no next-token target otherwise)");
  if (!layers || !lora) return fail(MEBP_EINVAL, "layers / lora array is NULL");
  if (!grads && cfg->lora_mask) return fail(MEBP_EINVAL, "grads array is NULL");
  for (int l = 0; l < cfg->n_layers; ++l) {
    if ((e = check_layer(cfg, l, &layers[l], &lora[l]))) return e;
    if ((e = check_grads(cfg, grads ? &grads[l] : nullptr))) return e;
  }
  if ((e = check_q4(emb, "embedding")) || (e = check_act(norm_final, "norm_final")) ||
      (e = check_ws(cfg, B, T, ws, ws_bytes)))
    return e;
  if (dx0 && !aligned(dx0, 16)) return fail(MEBP_EINVAL, "dx0 not 16-byte aligned");
  if (!ids || !aligned(ids, 4)) return fail(MEBP_EINVAL, "ids NULL or misaligned");
  if (!loss || !aligned(loss, 4)) return fail(MEBP_EINVAL, "loss NULL or misaligned");
  return MEBP_OK;
}

int mebp_train_step(const mebp_config* cfg, const mebp_q4* emb, const mebp_layer_base* layers,
                    const float* norm_final, const mebp_layer_lora* lora, const int32_t* ids, int32_t B, int32_t T,
                    float* ckpt, float* loss, const mebp_layer_lora_grad* grads, float* dx0, void* ws,
                    size_t ws_bytes, mebp_stream_t stream) {
  int e;
  if ((e = check_train_args(cfg, emb, layers, norm_final, lora, ids, B, T, loss, grads, dx0, ws, ws_bytes)) ||
      (e = check_act(ckpt, "ckpt")))
    return e;
  return guarded(cfg, B, T, ws, stream, [&] {
    return train_step_impl(cfg, emb, layers, norm_final, lora, ids, B, T, ckpt, nullptr, loss, grads, dx0, ws, stream);
  });
}

int mebp_train_step_offload(const mebp_config* cfg, const mebp_q4* emb, const mebp_layer_base* layers,
                            const float* norm_final, const mebp_layer_lora* lora, const int32_t* ids, int32_t B,
                            int32_t T, float* ckpt_host, float* ring, int32_t ring_slots, float* loss,
                            const mebp_layer_lora_grad* grads, float* dx0, void* ws, size_t ws_bytes,
                            mebp_stream_t stream) {
  int e;
  if ((e = check_train_args(cfg, emb, layers, norm_final, lora, ids, B, T, loss, grads, dx0, ws, ws_bytes)) ||
      (e = check_act(ring, "ring")))
    return e;
  if (ring_slots < 4 || ring_slots > MEBP_RING_MAX)
    return fail(MEBP_EINVAL, "ring_slots %d not in [4, %d]", ring_slots, MEBP_RING_MAX);
  if (!ckpt_host || !aligned(ckpt_host, 16)) return fail(MEBP_EINVAL, "ckpt_host NULL or not 16-byte aligned");
  hipPointerAttribute_t pa;
  if (hipPointerGetAttributes(&pa, ckpt_host) != hipSuccess || pa.type != hipMemoryTypeHost) {
    (void)hipGetLastError();
    return fail(MEBP_EINVAL, "ckpt_host is not pinned host memory (allocate it with hipHostMalloc)");
  }
  OffloadStreams* os = offload_streams();
  if (!os) return fail(MEBP_EHIP, "could not create the copy stream");
  Offload off;
  off.host = ckpt_host;
  // the device address of the pinned buffer, when the runtime reports it for exactly this
  // pointer and with the same alignment
  if (pa.hostPointer == (void*)ckpt_host && pa.devicePointer && aligned(pa.devicePointer, 16))
    off.host_dev = (float*)pa.devicePointer;
  off.R = ring_slots;
  off.cp = os->cp;
  off.ev_go = os->ev_go;
  for (int i = 0; i < MEBP_RING_MAX; ++i) {
    off.ev_in[i] = os->ev_in[i];
    off.ev_out[i] = os->ev_out[i];
  }
  static std::mutex mu;  // the copy stream and its events are shared by the calls on a device
  std::lock_guard<std::mutex> g(mu);
  return guarded(cfg, B, T, ws, stream, [&] {
    return train_step_impl(cfg, emb, layers, norm_final, lora, ids, B, T, ring, &off, loss, grads, dx0, ws, stream);
  });
}

int mebp_lora_grad_accumulate(const mebp_config* cfg, const mebp_layer_lora_grad* grads,
                              const mebp_layer_lora_grad* acc, float scale, int32_t first, mebp_stream_t stream) {
  int e;
  if ((e = check_config(cfg))) return e;
  if (!isfinite(scale)) return fail(MEBP_EINVAL, "scale is not finite");
  if (!cfg->lora_mask) return MEBP_OK;
  if (!grads || !acc) return fail(MEBP_EINVAL, "grads or acc array is NULL");
  const Dims D = dims(cfg, 1, 1);
  std::vector<OptSeg> segs;
  for (int l = 0; l < cfg->n_layers; ++l)
    for (int p = 0; p < MEBP_NPROJ; ++p) {
      if (!(cfg->lora_mask >> p & 1)) continue;
      const size_t n[2] = {(size_t)D.r * D.in[p], (size_t)D.out[p] * D.r};
      float* dst[2] = {acc[l].dA[p], acc[l].dB[p]};
      const float* src[2] = {grads[l].dA[p], grads[l].dB[p]};
      for (int k = 0; k < 2; ++k) {
        if (!dst[k] || !src[k]) return fail(MEBP_EINVAL, "layer %d %s: NULL tensor", l, kProjName[p]);
        if (!aligned(dst[k], 16) || !aligned(src[k], 16))
          return fail(MEBP_EINVAL, "layer %d %s: tensor not 16-byte aligned", l, kProjName[p]);
        segs.push_back(OptSeg{dst[k], src[k], nullptr, nullptr, (uint32_t)(n[k] / 4)});
      }
    }
  OptArgs a{};
  HIP_TRY(launch_lora_opt(segs.data(), (int)segs.size(), a, 1, scale, first ? 1 : 0, (hipStream_t)stream));
  return MEBP_OK;
}

int mebp_lora_adamw_step(const mebp_config* cfg, const mebp_layer_lora_state* params,
                         const mebp_layer_lora_grad* grads, const mebp_layer_lora_state* m,
                         const mebp_layer_lora_state* v, const mebp_adamw_hparams* hp, mebp_stream_t stream) {
  int e;
  if ((e = check_config(cfg))) return e;
  if (!hp) return fail(MEBP_EINVAL, "hparams is NULL");
  if (!isfinite(hp->lr) || !isfinite(hp->eps) || !isfinite(hp->weight_decay) || !isfinite(hp->grad_scale) ||
      !(hp->beta1 >= 0.f && hp->beta1 < 1.f) || !(hp->beta2 >= 0.f && hp->beta2 < 1.f) || hp->eps < 0.f)
    return fail(MEBP_EINVAL, "bad AdamW hyper-parameters");
  if (hp->step < 1) return fail(MEBP_EINVAL, "step %d < 1", hp->step);
  if (!cfg->lora_mask) return MEBP_OK;
  if (!params || !grads || !m || !v) return fail(MEBP_EINVAL, "params, grads, m or v array is NULL");
  const Dims D = dims(cfg, 1, 1);
  std::vector<OptSeg> segs;
  for (int l = 0; l < cfg->n_layers; ++l)
    for (int p = 0; p < MEBP_NPROJ; ++p) {
      if (!(cfg->lora_mask >> p & 1)) continue;
      const size_t n[2] = {(size_t)D.r * D.in[p], (size_t)D.out[p] * D.r};
      float* ps[2] = {params[l].A[p], params[l].B[p]};
      const float* gs[2] = {grads[l].dA[p], grads[l].dB[p]};
      float* ms[2] = {m[l].A[p], m[l].B[p]};
      float* vs[2] = {v[l].A[p], v[l].B[p]};
      for (int k = 0; k < 2; ++k) {
        if (!ps[k] || !gs[k] || !ms[k] || !vs[k]) return fail(MEBP_EINVAL, "layer %d %s: NULL tensor", l, kProjName[p]);
        if (!aligned(ps[k], 16) || !aligned(gs[k], 16) || !aligned(ms[k], 16) || !aligned(vs[k], 16))
          return fail(MEBP_EINVAL, "layer %d %s: tensor not 16-byte aligned", l, kProjName[p]);
        if ((const float*)ps[k] == gs[k] || ps[k] == ms[k] || ps[k] == vs[k] || ms[k] == vs[k])
          return fail(MEBP_EINVAL, "layer %d %s: aliased optimizer tensors", l, kProjName[p]);
        segs.push_back(OptSeg{ps[k], gs[k], ms[k], vs[k], (uint32_t)(n[k] / 4)});
      }
    }
  OptArgs a{};
  a.lr = hp->lr;
  a.beta1 = hp->beta1;
  a.beta2 = hp->beta2;
  a.eps = hp->eps;
  a.weight_decay = hp->weight_decay;
  a.grad_scale = hp->grad_scale;
  a.inv_bc1 = (float)(1.0 / (1.0 - pow((double)hp->beta1, (double)hp->step)));
  a.inv_bc2 = (float)(1.0 / (1.0 - pow((double)hp->beta2, (double)hp->step)));
  HIP_TRY(launch_lora_opt(segs.data(), (int)segs.size(), a, 0, 0.f, 0, (hipStream_t)stream));
  return MEBP_OK;
}

int mebp_dequant_q4(const mebp_q4* w, int32_t rows, int32_t cols, int32_t group, float* out_f32, uint16_t* out_bf16,
                    mebp_stream_t stream) {
  int e;
  if ((e = check_q4(w, "weight"))) return e;
  if (rows < 0 || cols < 0) return fail(MEBP_EINVAL, "negative size");
  if (cols % 8) return fail(MEBP_EUNSUPPORTED, "cols %d not a multiple of 8", cols);
  if (group != 32) return fail(MEBP_EUNSUPPORTED, "group %d != 32", group);
  if (!out_f32 && !out_bf16) return fail(MEBP_EINVAL, "no output requested");
  if ((out_f32 && !aligned(out_f32, 16)) || (out_bf16 && !aligned(out_bf16, 16)))
    return fail(MEBP_EINVAL, "outputs must be 16-byte aligned");
  HIP_TRY(launch_dequant(w->q4, w->scale, rows, cols, group, out_f32, out_bf16, (hipStream_t)stream));
  return MEBP_OK;
}

int mebp_test_gemm(int32_t kind, const mebp_q4* w, int32_t n_out, int32_t n_in, const void* x, int32_t M, float* out,
                   mebp_stream_t stream) {
  int e;
  if (kind < MEBP_TEST_GEMM_NT || kind > MEBP_TEST_GEMM_TN_BIG_W16) return fail(MEBP_EINVAL, "unknown GEMM kind %d", kind);
  if (kind == MEBP_TEST_GEMM_NT_LDS_W16 || kind == MEBP_TEST_GEMM_TN_BIG_W16) {
    if (!w || !w->q4 || !aligned(w->q4, 16)) return fail(MEBP_EINVAL, "16-bit weight NULL or not 16-byte aligned");
  } else if ((e = check_q4(w, "weight"))) {
    return e;
  }
  if (M < 1 || n_out < 1 || n_in < 1) return fail(MEBP_EINVAL, "non-positive size");
  if (M > 65536 || n_out > 65536 || n_in > 65536) return fail(MEBP_EUNSUPPORTED, "size above 65536");
  if (n_in % 16 || n_out % 16) return fail(MEBP_EUNSUPPORTED, "n_in %d / n_out %d not multiples of 16", n_in, n_out);
  if ((e = check_act(x, "x")) || (e = check_act(out, "out"))) return e;
  HIP_TRY(launch_gemm_probe(kind, w->q4, w->scale, n_out, n_in, x, M, out, (hipStream_t)stream));
  return MEBP_OK;
}

int mebp_kernel_timing(int32_t enable, int32_t capacity) {
  if (enable && capacity <= 0) return fail(MEBP_EINVAL, "capacity must be > 0");
  if (timing_enable(enable, capacity) != 0) return fail(MEBP_EHIP, "hipEventCreate failed");
  return MEBP_OK;
}

int mebp_kernel_repeat(const char* kernel, int32_t times) {
  if (set_repeat(kernel, times) != 0) return fail(MEBP_EINVAL, "kernel '%s' overwrites its own input and cannot be repeated", kernel);
  return MEBP_OK;
}

int mebp_kernel_timing_report(char* buf, size_t len) {
  const int n = timing_report(buf, len);
  if (n < 0) return fail(MEBP_EHIP, "event synchronisation failed");
  return n;
}

}  // extern "C"
