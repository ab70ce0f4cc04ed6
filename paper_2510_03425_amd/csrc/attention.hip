// Causal grouped-query attention with optional sliding window on gfx950, forward and
// backward, flash-style: scores never reach HBM; the forward keeps the row log-sum-exp
// for the backward. Softmax statistics are fp32. Activations q, k, v, O are fp16 and the
// score / output products run on fp16 MFMA; products with gradients (dO, dS) run on bf16
// MFMA with the activation operand converted to bf16 while it is staged.
//
// Layout trick used throughout: the 16x16 C tile of v_mfma_f32_16x16x32_bf16 gives lane l
// the rows 4*(l/16)+r (r = 0..3) of column l%16. Two such tiles stacked along the rows
// therefore hand lane l eight values of column l%16 at rows {4g..4g+3, 16+4g..16+4g+3}
// (g = l/16) -- exactly an MFMA operand for a 32-deep reduction over those rows, up to a
// fixed permutation of the reduction index. Softmax probabilities and their gradients are
// fed from registers into the next product this way; the other operand is read from an
// LDS tile stored reduction-contiguous (transposed at load time) with the same
// permutation (two 8-byte reads per lane).
//
//  forward : S^T = K Q^T (A = K rows from LDS, B = Q rows kept in registers);
//            O^T += V^T P^T (A = V^T from LDS, B = P from registers); row stats live in
//            the lane of their query, so rescaling needs no cross-lane traffic.
//  backward: the dK/dV kernels own a key block of one query head; with grouped-query
//            attention (or a split query loop) each stores fp32 partials and
//            k_attn_dkdv_reduce sums the heads of a group (and the chunks) in a fixed order.
//            The dQ kernel owns a query block. RoPE backward (rotation by minus the angle) is
//            applied where dK and dQ are finished, before the bf16 store.
#include <stdlib.h>

#include <algorithm>

#include "device_common.h"
#include "mebp_internal.h"

namespace mebp {
namespace {

constexpr float LOG2E = 1.4426950408889634f;

typedef uint16_t u16;

DEV uint4 load_frag_global(const void* p, bool ok) { return ok ? *(const uint4*)p : make_uint4(0, 0, 0, 0); }

// The causal window mask as one unsigned compare per element. Query i sees key j iff
// j <= i < T, j < T and (W == 0 or i - j < W): for a fixed query the visible keys form the
// range lo .. lo + span, and so do the visible queries of a fixed key. An empty range is
// lo = 2^30, span = 0 (x - lo is then negative, i.e. a huge unsigned value).
struct VisRange {
  int lo;
  uint32_t span;
};
DEV VisRange keys_of_query(int q, int T, int W) {
  if (q >= T) return {1 << 30, 0u};
  const int lo = W ? max(0, q - W + 1) : 0;
  return {lo, (uint32_t)(q - lo)};
}
DEV VisRange queries_of_key(int key, int T, int W) {
  if (key >= T) return {1 << 30, 0u};
  const int hi = W ? min(T - 1, key + W - 1) : T - 1;
  return {key, (uint32_t)(hi - key)};
}
DEV bool visible(const VisRange& v, int x) { return (uint32_t)(x - v.lo) <= v.span; }

// Buffer resource over the T rows of one sequence and one head (dh columns from `head0`
// elements into each row of pitch ld): loads past the last row return zero.
DEV rsrc_t seq_rsrc(const void* base, size_t row_first, int T, int ld, int head0, int dh) {
  return make_rsrc((const u16*)base + row_first * ld + head0, ((size_t)(T - 1) * ld + dh) * 2);
}

// Tile staging through registers: load() issues every global load of a tile at once (rows
// at or past `rows_ok` read as zero), the store functions write it to LDS. Kernels load
// the next tile before the products of the current one and store it after them, so the
// global-memory latency overlaps the MFMA work.
//
// Row chunks of an R x C tile of 16-bit values: chunk c is row c / (C/8), columns
// 8 (c % (C/8)) .. +8; thread t holds chunks t, t + NTH, ...
template <int R, int C, int NTH>
struct StageN {
  static constexpr int CH = C / 8, NC = R * CH, N = (NC + NTH - 1) / NTH;
  uint4 v[N];
  __device__ __forceinline__ void load(const u16* src, size_t ld, int rows_ok, int tid) {
#pragma unroll
    for (int i = 0; i < N; ++i) {
      const int c = tid + NTH * i, r = c / CH, col = (c % CH) * 8;
      v[i] = load_frag_global(src + (size_t)r * ld + col, c < NC && r < rows_ok);
    }
  }
  // The same tile through a buffer resource over the sequence's rows (rows past its end
  // read as zero) starting `row0` rows in: one per-lane offset and wave-uniform row
  // offsets, no per-load address arithmetic. Chunks past the tile (c >= NC) load rows of
  // the sequence that the store skips.
  __device__ __forceinline__ void load_rs(rsrc_t rs, int row0, int ld, int tid) {
    static_assert(NTH % CH == 0, "threads must cover whole rows");
    const uint32_t vo = (uint32_t)(((tid / CH) * ld + (tid % CH) * 8) * 2), rowB = (uint32_t)ld * 2;
#pragma unroll
    for (int i = 0; i < N; ++i) v[i] = bload128s(rs, vo, (uint32_t)(row0 + i * (NTH / CH)) * rowB);
  }
  // CONV: fp16 source values stored as bf16
  template <bool CONV>
  __device__ __forceinline__ void store(u16* dst, int LD, int tid) const {
#pragma unroll
    for (int i = 0; i < N; ++i) {
      const int c = tid + NTH * i, r = c / CH, col = (c % CH) * 8;
      if (c < NC) *(uint4*)(dst + r * LD + col) = CONV ? f16x8_to_bf16x8(v[i]) : v[i];
    }
  }
};

// 8 x 8 blocks of an R x C tile: block b covers rows 8 (b % RB) .. +8 and columns
// 8 (b / RB) .. +8, so one load feeds a row-major copy (store_n) and a transposed copy
// dst[col][row] (store_t) of the tile.
template <int R, int C, int NTH>
struct StageB {
  static constexpr int RB = R / 8, CB = C / 8, NB = RB * CB, N = (NB + NTH - 1) / NTH;
  uint4 v[N][8];
  __device__ __forceinline__ void load(const u16* src, size_t ld, int rows_ok, int tid) {
#pragma unroll
    for (int i = 0; i < N; ++i) {
      const int b = tid + NTH * i, rb = b % RB, cb = b / RB;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int r = rb * 8 + j;
        v[i][j] = load_frag_global(src + (size_t)r * ld + cb * 8, b < NB && r < rows_ok);
      }
    }
  }
  // buffer-resource form of load (see StageN::load_rs)
  __device__ __forceinline__ void load_rs(rsrc_t rs, int row0, int ld, int tid) {
    const uint32_t rowB = (uint32_t)ld * 2;
#pragma unroll
    for (int i = 0; i < N; ++i) {
      const int b = min(tid + NTH * i, NB - 1), rb = b % RB, cb = b / RB;
      const uint32_t vo = (uint32_t)(((rb * 8) * ld + cb * 8) * 2);
#pragma unroll
      for (int j = 0; j < 8; ++j) v[i][j] = bload128s(rs, vo, (uint32_t)(row0 + j) * rowB);
    }
  }
  template <bool CONV>
  __device__ __forceinline__ void store_n(u16* dst, int LD, int tid) const {
#pragma unroll
    for (int i = 0; i < N; ++i) {
      const int b = tid + NTH * i, rb = b % RB, cb = b / RB;
      if (b >= NB) continue;
#pragma unroll
      for (int j = 0; j < 8; ++j) *(uint4*)(dst + (rb * 8 + j) * LD + cb * 8) = CONV ? f16x8_to_bf16x8(v[i][j]) : v[i][j];
    }
  }
  template <bool CONV>
  __device__ __forceinline__ void store_t(u16* dst, int LD, int tid) const {
#pragma unroll
    for (int i = 0; i < N; ++i) {
      const int b = tid + NTH * i, rb = b % RB, cb = b / RB;
      if (b >= NB) continue;
      uint32_t in[8][4];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const uint4 x = CONV ? f16x8_to_bf16x8(v[i][j]) : v[i][j];
        in[j][0] = x.x; in[j][1] = x.y; in[j][2] = x.z; in[j][3] = x.w;
      }
#pragma unroll
      for (int jc = 0; jc < 8; ++jc) {
        const int d = jc >> 1;
        uint4 o;
        if (jc & 1) {
          o = make_uint4(perm_hi16(in[0][d], in[1][d]), perm_hi16(in[2][d], in[3][d]), perm_hi16(in[4][d], in[5][d]),
                         perm_hi16(in[6][d], in[7][d]));
        } else {
          o = make_uint4(perm_lo16(in[0][d], in[1][d]), perm_lo16(in[2][d], in[3][d]), perm_lo16(in[4][d], in[5][d]),
                         perm_lo16(in[6][d], in[7][d]));
        }
        // two 8-byte stores: transposed rows are padded by 4 halves (8-byte aligned), which
        // keeps the 8-byte fragment reads of 16 consecutive rows on distinct banks
        uint2* dt = (uint2*)(dst + (cb * 8 + jc) * LD + rb * 8);
        dt[0] = make_uint2(o.x, o.y);
        dt[1] = make_uint2(o.z, o.w);
      }
    }
  }
};

// A/B fragment from an LDS tile stored [row][k] (k contiguous): lane l reads
// row row0 + l%16, k0 + 8*(l/16) .. +8.
DEV uint4 frag_rows(const u16* s, int ld, int row0, int k0, int lane) {
  return *(const uint4*)(s + (row0 + (lane & 15)) * ld + k0 + 8 * (lane >> 4));
}
// Permuted fragment: row row0 + l%16, columns c0 + 4g .. +4 and c0 + 16 + 4g .. +4.
DEV uint4 frag_perm(const u16* s, int ld, int row0, int c0, int lane) {
  const u16* p = s + (row0 + (lane & 15)) * ld + c0 + 4 * (lane >> 4);
  const uint2 a = *(const uint2*)p, b = *(const uint2*)(p + 16);
  return make_uint4(a.x, a.y, b.x, b.y);
}
// Pack two C tiles (8 floats: tile0 rows r=0..3, tile1 rows r=0..3) into an operand.
template <class Op>
DEV uint4 pack_frag(const f32x4& t0, const f32x4& t1) {
  return make_uint4(Op::pack(t0[0], t0[1]), Op::pack(t0[2], t0[3]), Op::pack(t1[0], t1[1]), Op::pack(t1[2], t1[3]));
}
// Tile of this workgroup: (query or key block [x chunk], head, sequence). Unsplit grids (long
// sequences) use the XCD-aware order, so that the blocks of one head, which read the same
// K/V (or Q/dO) rows, share an L2; split grids keep the plain order.
DEV TileId attn_tile(int nck) {
  if (nck) return TileId{(int)blockIdx.x, (int)blockIdx.y, (int)blockIdx.z};
  return xcd_tile();
}

// ------------------------------------------------------------------------------ forward
// 64 queries (4 waves of 16) of one head per workgroup, 64-key blocks. With `nck` > 0 the
// key range of the query tile is split into chunks of `ck` keys, one per workgroup
// (blockIdx.x = tile * nck + chunk): short sequences then still give enough workgroups
// to fill the chip. A chunk stores its unnormalised output and its row statistics
// (max, sum, base-2 domain) in fp32 and k_attn_fwd_combine merges the chunks in order.
template <int DH>
__global__ __launch_bounds__(256) void k_attn_fwd(const AttnArgs a, float* part, int nck, int ck) {
  constexpr int KB = 64, LDK = DH + 8, LDV = KB + 4, NKS = DH / 32, NT = DH / 16;
  __shared__ __attribute__((aligned(16))) u16 Ks[KB * LDK];
  __shared__ __attribute__((aligned(16))) u16 Vt[DH * LDV];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const TileId id = attn_tile(nck);
  const int tile = nck ? id.x / nck : id.x, chunk = nck ? id.x % nck : 0;
  const int T = a.T, h = id.y, b = id.z, grp = a.Hq / a.Hkv, kvh = h / grp;
  const int q0 = tile * 64, qw = q0 + 16 * w, q = qw + (lane & 15);
  const VisRange kvis = keys_of_query(q, a.T, a.window);
  const float sc = LOG2E / sqrtf((float)DH);
  const size_t rowb = (size_t)b * T;

  int kv_lo = 0;
  if (a.window) kv_lo = max(0, q0 - a.window + 1) & ~(KB - 1);
  int kv_hi = min(T, q0 + 64);
  if (nck) {
    kv_lo += chunk * ck;
    if (kv_lo >= kv_hi) return;  // the whole workgroup: no chunk here
    kv_hi = min(kv_hi, kv_lo + ck);
  }

  StageN<KB, DH, 256> kst;  // K row-major (A operand of S^T = K Q^T)
  StageB<KB, DH, 256> vst;  // V, stored transposed (A operand of O^T += V^T P^T)
  const rsrc_t rK = seq_rsrc(a.k, rowb, T, a.ldk, kvh * DH, DH), rV = seq_rsrc(a.v, rowb, T, a.ldk, kvh * DH, DH);
  auto gload = [&](int kv0) {
    kst.load_rs(rK, kv0, a.ldk, tid);
    vst.load_rs(rV, kv0, a.ldk, tid);
  };
  gload(kv_lo);

  uint4 qf[NKS];
#pragma unroll
  for (int ks = 0; ks < NKS; ++ks)
    qf[ks] = load_frag_global(a.q + (rowb + q) * a.ldq + h * DH + 32 * ks + 8 * (lane >> 4), q < T);
  f32x4 oacc[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) oacc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_i = -1e30f, l_i = 0.f;

  for (int kv0 = kv_lo; kv0 < kv_hi; kv0 += KB) {
    __syncthreads();  // every wave is done with the previous block's tiles
    kst.template store<false>(Ks, LDK, tid);
    vst.template store_t<false>(Vt, LDV, tid);
    __syncthreads();
    if (kv0 + KB < kv_hi) gload(kv0 + KB);  // next block in flight during this one
    f32x4 s[4];
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) {
      s[kt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks)
        s[kt] = mfma16_raw<OpF16>(frag_rows(Ks, LDK, kt * 16, ks * 32, lane), qf[ks], s[kt]);
    }
    float mloc = -1e30f;
#pragma unroll
    for (int kt = 0; kt < 4; ++kt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const bool vis = visible(kvis, kv0 + kt * 16 + 4 * (lane >> 4) + r);
        const float v = vis ? s[kt][r] * sc : -INFINITY;
        s[kt][r] = v;
        mloc = fmaxf(mloc, v);
      }
    mloc = fmaxf(mloc, __shfl_xor(mloc, 16, 64));
    mloc = fmaxf(mloc, __shfl_xor(mloc, 32, 64));
    const float m_new = fmaxf(m_i, mloc);
    const float alpha = exp2_fast(m_i - m_new);
    float ls = 0.f;
#pragma unroll
    for (int kt = 0; kt < 4; ++kt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float p = exp2_fast(s[kt][r] - m_new);
        s[kt][r] = p;
        ls += p;
      }
    ls += __shfl_xor(ls, 16, 64);
    ls += __shfl_xor(ls, 32, 64);
    l_i = l_i * alpha + ls;
    m_i = m_new;
#pragma unroll
    for (int t = 0; t < NT; ++t) oacc[t] *= alpha;
#pragma unroll
    for (int kp = 0; kp < 2; ++kp) {
      const uint4 pf = pack_frag<OpF16>(s[2 * kp], s[2 * kp + 1]);
#pragma unroll
      for (int t = 0; t < NT; ++t) oacc[t] = mfma16_raw<OpF16>(frag_perm(Vt, LDV, t * 16, kp * 32, lane), pf, oacc[t]);
    }
  }
  if (q >= T) return;
  if (nck) {
    // chunk partial: [B][Hq][nck][T][DH] unnormalised output, then [B][Hq][nck][T] (max, sum)
    const size_t pr = (((size_t)b * a.Hq + h) * nck + chunk) * T + q;
    float* op = part + pr * DH;
#pragma unroll
    for (int t = 0; t < NT; ++t)
      *(float4*)(op + t * 16 + 4 * (lane >> 4)) = make_float4(oacc[t][0], oacc[t][1], oacc[t][2], oacc[t][3]);
    if ((lane >> 4) == 0)
      ((float2*)(part + (size_t)a.B * a.Hq * nck * T * DH))[pr] = make_float2(m_i, l_i);
    return;
  }
  const float inv = 1.0f / l_i;
  f16* orow = a.o + (rowb + q) * a.ldq + h * DH;
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    const int e = t * 16 + 4 * (lane >> 4);
    *(uint2*)(orow + e) = make_uint2(pack_f16x2(oacc[t][0] * inv, oacc[t][1] * inv),
                                     pack_f16x2(oacc[t][2] * inv, oacc[t][3] * inv));
  }
  if ((lane >> 4) == 0) a.lse[((size_t)b * a.Hq + h) * T + q] = (m_i + log2f(l_i)) / LOG2E;
}

// Number of key chunks of `ck` keys that query tile `tile` (64 queries) of k_attn_fwd and
// k_attn_bwd_dq visits (key blocks of KB, aligned as in those kernels).
__host__ __device__ inline int fwd_tile_chunks(int tile, int T, int window, int KB, int ck) {
  const int q0 = tile * 64;
  const int lo = window ? (q0 - window + 1 > 0 ? q0 - window + 1 : 0) & ~(KB - 1) : 0;
  const int hi = T < q0 + 64 ? T : q0 + 64;
  return hi > lo ? (hi - lo + ck - 1) / ck : 0;
}

// Merge of the key chunks of k_attn_fwd: O = sum_c 2^(m_c - M) O_c / sum_c 2^(m_c - M) l_c
// with M = max_c m_c, chunks in order; also the row log-sum-exp. One thread per (batch,
// head, query, 8 columns).
template <int DH>
__global__ void k_attn_fwd_combine(const AttnArgs a, const float* part, int nck, int ck) {
  constexpr int G = DH / 8;
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int T = a.T;
  if (i >= (size_t)a.B * a.Hq * T * G) return;
  const int g = (int)(i % G);
  const size_t row = i / G;  // (b * Hq + h) * T + q
  const int q = (int)(row % T);
  const size_t bh = row / T;
  const int h = (int)(bh % a.Hq), b = (int)(bh / a.Hq);
  const int n = fwd_tile_chunks(q / 64, T, a.window, 64, ck);
  const float2* ml = (const float2*)(part + (size_t)a.B * a.Hq * nck * T * DH);
  float M = -1e30f;
  for (int c = 0; c < n; ++c) M = fmaxf(M, ml[(bh * nck + c) * T + q].x);
  float L = 0.f, acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  for (int c = 0; c < n; ++c) {
    const size_t pr = (bh * nck + c) * T + q;
    const float2 st = ml[pr];
    const float wgt = exp2_fast(st.x - M);
    L += wgt * st.y;
    const float4 x0 = *(const float4*)(part + pr * DH + 8 * g), x1 = *(const float4*)(part + pr * DH + 8 * g + 4);
    acc[0] += wgt * x0.x; acc[1] += wgt * x0.y; acc[2] += wgt * x0.z; acc[3] += wgt * x0.w;
    acc[4] += wgt * x1.x; acc[5] += wgt * x1.y; acc[6] += wgt * x1.z; acc[7] += wgt * x1.w;
  }
  const float inv = 1.0f / L;
  f16* orow = a.o + ((size_t)b * T + q) * a.ldq + h * DH + 8 * g;
  *(uint4*)orow = make_uint4(pack_f16x2(acc[0] * inv, acc[1] * inv), pack_f16x2(acc[2] * inv, acc[3] * inv),
                             pack_f16x2(acc[4] * inv, acc[5] * inv), pack_f16x2(acc[6] * inv, acc[7] * inv));
  if (g == 0) a.lse[row] = (M + log2f(L)) / LOG2E;
}

// ------------------------------------------------------------- forward, 32-query waves
// For longer sequences: every wave owns 32 queries and uses v_mfma_f32_32x32x16_f16, so
// each K / V^T fragment read from LDS feeds twice the MACs of the 16-query kernel above.
// S^T = K Q^T puts one query per lane column (keys 8(r/4)+4h+r%4 of a 32-key tile in lane
// register r, h = lane/32), so the row statistics need one cross-lane exchange (lane^32)
// and O^T's rescaling is lane-local. P^T enters O^T += V^T P^T straight from registers as
// the B operand: registers 0..7 (then 8..15) of an S^T tile are the keys
// {4h..4h+3, 8+4h..8+4h+3} of a 16-key step, and the V^T fragment is read with the same
// key order (two 8-byte LDS reads). The next K / V block is loaded into registers while
// the current one is multiplied.
typedef float f32x16 __attribute__((ext_vector_type(16)));
DEV f32x16 mfma32_f16(uint4 a, uint4 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
}

DEV f32x16 mfma32_bf16(uint4 a, uint4 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c, 0, 0,
                                                 0);
}

// x += sum_i A_i B_i over N MFMAs whose A fragments are 16-byte LDS reads at p + 16 i (halves):
// each read is issued FA MFMAs ahead of its use (scheduling groups keep the compiler from
// moving it next to the MFMA), so that no MFMA waits for the round trip of its own read
template <int FA, int N, class MF>
DEV f32x16 lds_chain(const u16* p, const uint4 (&b)[N], f32x16 x, MF mf) {
  uint4 buf[FA + 2];
#pragma unroll
  for (int i = 0; i < FA; ++i) buf[i] = *(const uint4*)(p + 16 * i);
#pragma unroll
  for (int i = 0; i < N; ++i) {
    if (i + FA < N) buf[(i + FA) % (FA + 2)] = *(const uint4*)(p + 16 * (i + FA));
    x = mf(buf[i % (FA + 2)], b[i], x);
  }
  __builtin_amdgcn_sched_group_barrier(0x100, FA, 0);
#pragma unroll
  for (int i = 0; i < N; ++i) {
    if (i + FA < N) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
  }
  return x;
}

template <int DH, int NW>
__global__ __launch_bounds__(64 * NW) void k_attn_fwd32(const AttnArgs a) {
  // V^T rows of 68 halves (34 dwords): the 16 lanes of one 8-byte LDS read cycle (16
  // consecutive rows) then fall on 32 distinct banks (with 72 halves, rows r and r + 8 shared
  // a bank: a 2-way conflict on every V^T fragment read)
  constexpr int NTH = 64 * NW, KB = 64, LDK = DH + 8, LDV = KB + 4;
  constexpr int FA = 3;  // LDS fragment reads in flight ahead of the MFMAs
  constexpr int NKS = DH / 16, NTO = DH / 32;
  constexpr int KCH = KB * DH / 8 / NTH;                // K chunks (8 halves) per thread
  constexpr int NVB = (KB / 8) * (DH / 8);               // 8x8 blocks of the V tile
  constexpr int VBL = (NVB + NTH - 1) / NTH;             // per thread (threads past NVB idle)
  static_assert(KCH >= 1 && KB * DH / 8 % NTH == 0, "K tile does not divide over the threads");
  __shared__ __attribute__((aligned(16))) u16 Ks[KB * LDK];
  __shared__ __attribute__((aligned(16))) u16 Vt[DH * LDV];
  const int tid = threadIdx.x, lane = tid & 63, w = __builtin_amdgcn_readfirstlane(tid >> 6), hl = lane >> 5;
  const TileId id = attn_tile(0);
  const int T = a.T, h = id.y, b = id.z, grp = a.Hq / a.Hkv, kvh = h / grp;
  const int q0 = id.x * (32 * NW), qw = q0 + 32 * w, q = qw + (lane & 31);
  const float sc = LOG2E / sqrtf((float)DH);
  const size_t rowb = (size_t)b * T;

  uint4 qf[NKS];
#pragma unroll
  for (int ks = 0; ks < NKS; ++ks)
    qf[ks] = load_frag_global(a.q + (rowb + q) * a.ldq + h * DH + 16 * ks + 8 * hl, q < T);
  f32x16 oacc[NTO];
#pragma unroll
  for (int t = 0; t < NTO; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[t][r] = 0.f;
  float m_i = -1e30f, l_i = 0.f;

  int kv_lo = 0;
  if (a.window) kv_lo = max(0, q0 - a.window + 1) & ~(KB - 1);
  const int kv_hi = min(T, q0 + 32 * NW);
  // wave's own visible key range (for skipping fully masked blocks)
  const int w_lo = a.window ? max(0, qw - a.window + 1) : 0, w_hi = min(T, qw + 32) - 1;
  const VisRange kvis = keys_of_query(q, T, a.window);

  uint4 kr[KCH], vr[VBL][8];
  // K / V rows of this sequence and KV head as buffer resources: rows past T read as zero;
  // each load is one per-lane offset fixed for the kernel plus a wave-uniform row offset
  const size_t kvbytes = ((size_t)(T - 1) * a.ldk + DH) * 2;
  const rsrc_t rK = make_rsrc((const u16*)a.k + rowb * a.ldk + kvh * DH, kvbytes);
  const rsrc_t rV = make_rsrc((const u16*)a.v + rowb * a.ldk + kvh * DH, kvbytes);
  const uint32_t rowB = (uint32_t)a.ldk * 2;
  // K: chunk c = tid + NTH i is row c / (DH/8) = tid / (DH/8) + i NTH / (DH/8), column (c % (DH/8)) 8
  const uint32_t offK = (uint32_t)(((tid / (DH / 8)) * a.ldk + (tid % (DH / 8)) * 8) * 2);
  // V: block bl = tid + NTH i, rows 8 (bl % (KB/8)) + j, columns 8 (bl / (KB/8))
  uint32_t offV[VBL];
#pragma unroll
  for (int i = 0; i < VBL; ++i) {
    const int bl = min(tid + NTH * i, NVB - 1);
    offV[i] = (uint32_t)((((bl % (KB / 8)) * 8) * a.ldk + (bl / (KB / 8)) * 8) * 2);
  }
  auto gload = [&](int kv0) {
    const uint32_t s0 = (uint32_t)kv0 * rowB;
#pragma unroll
    for (int i = 0; i < KCH; ++i) kr[i] = bload128s(rK, offK, s0 + (uint32_t)(i * (NTH / (DH / 8))) * rowB);
#pragma unroll
    for (int i = 0; i < VBL; ++i)
#pragma unroll
      for (int j = 0; j < 8; ++j) vr[i][j] = bload128s(rV, offV[i], s0 + (uint32_t)j * rowB);
  };
  auto sstore = [&]() {
#pragma unroll
    for (int i = 0; i < KCH; ++i) {
      const int c = tid + NTH * i, r = c / (DH / 8), col = (c % (DH / 8)) * 8;
      *(uint4*)(Ks + r * LDK + col) = kr[i];
    }
#pragma unroll
    for (int i = 0; i < VBL; ++i) {
      const int bl = tid + NTH * i, rb = bl % (KB / 8), cb = bl / (KB / 8);
      if (bl >= NVB) continue;
      const uint32_t* in = (const uint32_t*)vr[i];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int d = j >> 1;
        uint4 o;
        if (j & 1) {
          o.x = perm_hi16(in[0 * 4 + d], in[1 * 4 + d]);
          o.y = perm_hi16(in[2 * 4 + d], in[3 * 4 + d]);
          o.z = perm_hi16(in[4 * 4 + d], in[5 * 4 + d]);
          o.w = perm_hi16(in[6 * 4 + d], in[7 * 4 + d]);
        } else {
          o.x = perm_lo16(in[0 * 4 + d], in[1 * 4 + d]);
          o.y = perm_lo16(in[2 * 4 + d], in[3 * 4 + d]);
          o.z = perm_lo16(in[4 * 4 + d], in[5 * 4 + d]);
          o.w = perm_lo16(in[6 * 4 + d], in[7 * 4 + d]);
        }
        // 8-byte aligned rows: two 8-byte stores
        uint2* dv = (uint2*)(Vt + (cb * 8 + j) * LDV + rb * 8);
        dv[0] = make_uint2(o.x, o.y);
        dv[1] = make_uint2(o.z, o.w);
      }
    }
  };

  if (kv_lo < kv_hi) gload(kv_lo);
  for (int kv0 = kv_lo; kv0 < kv_hi; kv0 += KB) {
    __syncthreads();  // every wave is done with the previous block's tiles
    sstore();
    __syncthreads();
    if (kv0 + KB < kv_hi) gload(kv0 + KB);  // next block in flight during this one
    if (kv0 > w_hi || kv0 + KB - 1 < w_lo) continue;  // nothing visible for this wave
    f32x16 s[2];
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int r = 0; r < 16; ++r) s[kt][r] = 0.f;
    {
      // the 2 x NKS score MFMAs in (key tile, depth) order, each K fragment read from LDS FA
      // MFMAs ahead of its use, so that no MFMA waits for the round trip of its own read
      // (the scheduling groups keep the compiler from moving the reads next to their use;
      // alternating the two key tiles' chains measured 3 % slower)
      constexpr int NR = 2 * NKS;
      uint4 kb[FA + 2];
      auto rdk = [&](int i) {
        return *(const uint4*)(Ks + ((i / NKS) * 32 + (lane & 31)) * LDK + 8 * hl + 16 * (i % NKS));
      };
#pragma unroll
      for (int i = 0; i < FA; ++i) kb[i] = rdk(i);
#pragma unroll
      for (int i = 0; i < NR; ++i) {
        if (i + FA < NR) kb[(i + FA) % (FA + 2)] = rdk(i + FA);
        s[i / NKS] = mfma32_f16(kb[i % (FA + 2)], qf[i % NKS], s[i / NKS]);
      }
      __builtin_amdgcn_sched_group_barrier(0x100, FA, 0);
#pragma unroll
      for (int i = 0; i < NR; ++i) {
        if (i + FA < NR) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      }
    }
    float mloc = -1e30f;
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const bool vis = visible(kvis, kv0 + kt * 32 + 8 * (r >> 2) + 4 * hl + (r & 3));
        const float v = vis ? s[kt][r] * sc : -INFINITY;
        s[kt][r] = v;
        mloc = fmaxf(mloc, v);
      }
    mloc = fmaxf(mloc, __shfl_xor(mloc, 32, 64));
    // The running maximum only moves when a row's block maximum exceeds it by more than
    // 2^8 (base-2 domain): the probabilities stay below 256 and the sum and the output are
    // both taken relative to the same stale maximum, so the result is unchanged; most
    // blocks then skip the rescale of the output accumulators.
    const float m_new = mloc > m_i + 8.f ? mloc : m_i;
    float ls = 0.f;
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float p = exp2_fast(s[kt][r] - m_new);
        s[kt][r] = p;
        ls += p;
      }
    ls += __shfl_xor(ls, 32, 64);
    if (__builtin_amdgcn_ballot_w64(m_new != m_i)) {
      const float alpha = exp2_fast(m_i - m_new);
      l_i *= alpha;
#pragma unroll
      for (int t = 0; t < NTO; ++t) oacc[t] *= alpha;
    }
    l_i += ls;
    m_i = m_new;
    {
      // O^T += V^T P^T: 4 x NTO MFMAs in (key step, output tile) order, the V^T fragments read
      // FA MFMAs ahead as above
      constexpr int NPV = 4 * NTO;
      uint4 pf[4];
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        const f32x16& st = s[kk >> 1];
        const int r0 = 8 * (kk & 1);
        pf[kk] = make_uint4(pack_f16x2(st[r0 + 0], st[r0 + 1]), pack_f16x2(st[r0 + 2], st[r0 + 3]),
                            pack_f16x2(st[r0 + 4], st[r0 + 5]), pack_f16x2(st[r0 + 6], st[r0 + 7]));
      }
      uint4 vb[FA + 2];
      auto rdv = [&](int i) {
        const u16* vp = Vt + ((i % NTO) * 32 + (lane & 31)) * LDV + (i / NTO) * 16 + 4 * hl;
        const uint2 x0 = *(const uint2*)vp, x1 = *(const uint2*)(vp + 8);
        return make_uint4(x0.x, x0.y, x1.x, x1.y);
      };
#pragma unroll
      for (int i = 0; i < FA; ++i) vb[i] = rdv(i);
#pragma unroll
      for (int i = 0; i < NPV; ++i) {
        if (i + FA < NPV) vb[(i + FA) % (FA + 2)] = rdv(i + FA);
        oacc[i % NTO] = mfma32_f16(vb[i % (FA + 2)], pf[i / NTO], oacc[i % NTO]);
      }
      __builtin_amdgcn_sched_group_barrier(0x100, FA, 0);
#pragma unroll
      for (int i = 0; i < NPV; ++i) {
        if (i + FA < NPV) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      }
    }
  }
  if (q < T) {
    const float inv = 1.0f / l_i;
    f16* orow = a.o + (rowb + q) * a.ldq + h * DH;
#pragma unroll
    for (int t = 0; t < NTO; ++t)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int e = t * 32 + 8 * g + 4 * hl;
        *(uint2*)(orow + e) = make_uint2(pack_f16x2(oacc[t][4 * g] * inv, oacc[t][4 * g + 1] * inv),
                                         pack_f16x2(oacc[t][4 * g + 2] * inv, oacc[t][4 * g + 3] * inv));
      }
    if (hl == 0) a.lse[((size_t)b * a.Hq + h) * T + q] = (m_i + log2f(l_i)) / LOG2E;
  }
}

// ------------------------------------------------------------------------------ backward
// delta[b][h][t] = sum_e dO[b*T+t][h*dh+e] * O[b*T+t][h*dh+e]
// One thread per (row, head, 8 columns); the dh/8 threads of a (row, head) are
// consecutive lanes of one wave and combine their sums with butterfly shuffles.
__global__ void k_attn_delta(const bf16* dO, const f16* O, int ld, int B, int T, int H, int dh, float* delta) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int G = dh / 8;
  const bool ok = i < (size_t)B * T * H * G;
  const int c = (int)(i % G);
  const size_t rh = i / G;
  const int h = (int)(rh % H);
  const size_t row = rh / H;
  float acc = 0.f;
  if (ok) {
    const uint4 x = *(const uint4*)(dO + row * ld + h * dh + 8 * c), y = *(const uint4*)(O + row * ld + h * dh + 8 * c);
    const uint32_t* xp = (const uint32_t*)&x;
    const uint32_t* yp = (const uint32_t*)&y;
#pragma unroll
    for (int j = 0; j < 4; ++j) acc += bf16_lo(xp[j]) * f16_lo(yp[j]) + bf16_hi(xp[j]) * f16_hi(yp[j]);
  }
  for (int m = 1; m < G; m <<= 1) acc += __shfl_xor(acc, m, 64);
  if (ok && c == 0) {
    const int b = (int)(row / T), t = (int)(row % T);
    delta[((size_t)b * H + h) * T + t] = acc;
  }
}

// dK, dV for a block of 64 keys (4 waves of 16) and one query head. The workgroup walks
// the query tiles (QB queries) that can see its keys; with `nck` > 0 that query range is
// split into chunks of `cq` queries, one per workgroup (blockIdx.x = key block * nck +
// chunk). Partial results: with grouped-query attention, or with chunks, each workgroup
// stores fp32 partial dK / dV and k_attn_dkdv_reduce sums them in (chunk, head) order
// (deterministic); otherwise the epilogue finishes dK (scale, RoPE backward) and dV itself.
template <int DH, int QB>
__global__ __launch_bounds__(256) void k_attn_bwd_dkdv(const AttnArgs a, float* part, int nck, int cq) {
  constexpr int LDN = DH + 8, LDT_ = QB + 8, NKS = DH / 32, NT = DH / 16, NQT = QB / 16;
  __shared__ __attribute__((aligned(16))) u16 Qs[QB * LDN];   // fp16 (scores)
  __shared__ __attribute__((aligned(16))) u16 dOs[QB * LDN];  // bf16
  __shared__ __attribute__((aligned(16))) u16 Qt[DH * LDT_];  // bf16 (dK product)
  __shared__ __attribute__((aligned(16))) u16 dOt[DH * LDT_]; // bf16
  __shared__ float lse_s[QB], del_s[QB];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const TileId id = attn_tile(nck);
  const int kblk = nck ? id.x / nck : id.x, chunk = nck ? id.x % nck : 0;
  const int T = a.T, h = id.y, b = id.z, grp = a.Hq / a.Hkv, kvh = h / grp, hh = h % grp;
  const int k0 = kblk * 64, kw = k0 + 16 * w, key = kw + (lane & 15);
  const VisRange qvis = queries_of_key(key, T, a.window);
  const float sc = LOG2E / sqrtf((float)DH);
  const size_t rowb = (size_t)b * T;

  int q_lo = k0 & ~(QB - 1);
  int q_hi = T;
  if (a.window) q_hi = min(T, k0 + 64 + a.window - 1);
  if (nck) {
    q_lo += chunk * cq;
    if (q_lo >= q_hi) return;  // the whole workgroup: no chunk here
    q_hi = min(q_hi, q_lo + cq);
  }

  StageB<QB, DH, 256> qst, dst;  // Q and dO tiles: row-major and transposed LDS copies
  const rsrc_t rQ = seq_rsrc(a.q, rowb, T, a.ldq, h * DH, DH), rdO = seq_rsrc(a.dO, rowb, T, a.ldq, h * DH, DH);
  float st_lse = 0.f, st_del = 0.f;
  const size_t stat0 = ((size_t)b * a.Hq + h) * T;  // this (sequence, head)'s row statistics
  const rsrc_t rL = make_rsrc(a.lse + stat0, (size_t)T * 4), rD = make_rsrc(a.delta + stat0, (size_t)T * 4);
  auto gload = [&](int qb0) {
    qst.load_rs(rQ, qb0, a.ldq, tid);
    dst.load_rs(rdO, qb0, a.ldq, tid);
    // the row statistics of queries qb0 + tid (tid < QB) through buffer loads, without a
    // branch, and scaled only when stored: a use right after the load would make the wave wait
    // for it, and so for every tile load issued before it
    {
      const int qq = qb0 + tid;
      const uint32_t so = (tid < QB && qq < T) ? (uint32_t)qq * 4 : 0x80000000u;
      st_lse = __uint_as_float(bload32(rL, so));
      st_del = __uint_as_float(bload32(rD, so));
    }
  };
  gload(q_lo);

  uint4 kf[NKS], vf[NKS];  // K fp16 (scores), V converted to bf16 (dP = dO V^T)
#pragma unroll
  for (int ks = 0; ks < NKS; ++ks) {
    const size_t off = (rowb + key) * a.ldk + kvh * DH + 32 * ks + 8 * (lane >> 4);
    kf[ks] = load_frag_global(a.k + off, key < T);
    vf[ks] = f16x8_to_bf16x8(load_frag_global(a.v + off, key < T));
  }
  f32x4 dk[NT], dv[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    dk[t] = f32x4{0.f, 0.f, 0.f, 0.f};
    dv[t] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  for (int qb0 = q_lo; qb0 < q_hi; qb0 += QB) {
    __syncthreads();  // every wave is done with the previous tile
    qst.template store_n<false>(Qs, LDN, tid);
    qst.template store_t<true>(Qt, LDT_, tid);
    dst.template store_n<false>(dOs, LDN, tid);
    dst.template store_t<false>(dOt, LDT_, tid);
    if (tid < QB) {
      lse_s[tid] = st_lse * LOG2E;
      del_s[tid] = st_del;
    }
    __syncthreads();
    // next tile in flight during this one; issued after the last tile too (rows past T read as
    // zero, rows past the range are unused), since loads behind a branch leave the compiler
    // only a full wait for them before the next MFMA
    gload(qb0 + QB);
    f32x4 s[NQT], dp[NQT];
#pragma unroll
    for (int qt = 0; qt < NQT; ++qt) {
      s[qt] = f32x4{0.f, 0.f, 0.f, 0.f};
      dp[qt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks) {
        s[qt] = mfma16_raw<OpF16>(frag_rows(Qs, LDN, qt * 16, ks * 32, lane), kf[ks], s[qt]);
        dp[qt] = mfma16_raw<OpBF16>(frag_rows(dOs, LDN, qt * 16, ks * 32, lane), vf[ks], dp[qt]);
      }
    }
#pragma unroll
    for (int qt = 0; qt < NQT; ++qt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int ql = qt * 16 + 4 * (lane >> 4) + r;
        const bool vis = visible(qvis, qb0 + ql);
        const float p = vis ? exp2_fast(s[qt][r] * sc - lse_s[ql]) : 0.f;
        s[qt][r] = p;
        dp[qt][r] = p * (dp[qt][r] - del_s[ql]);
      }
#pragma unroll
    for (int qp = 0; qp < NQT / 2; ++qp) {
      const uint4 pf = pack_frag<OpBF16>(s[2 * qp], s[2 * qp + 1]);
      const uint4 df = pack_frag<OpBF16>(dp[2 * qp], dp[2 * qp + 1]);
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        dv[t] = mfma16_raw<OpBF16>(pf, frag_perm(dOt, LDT_, t * 16, qp * 32, lane), dv[t]);
        dk[t] = mfma16_raw<OpBF16>(df, frag_perm(Qt, LDT_, t * 16, qp * 32, lane), dk[t]);
      }
    }
  }
  // epilogue: lane holds rows key kw + 4g + r, column e = 16t + lane%16
  if (grp > 1 || nck) {
    // fp32 partials, planes [chunk][dk: heads of the group, dv: heads of the group]
    const size_t plane = (size_t)a.B * T * a.Hkv * DH;
    float* base = part + (size_t)chunk * 2 * grp * plane;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int kk = kw + 4 * (lane >> 4) + r;
      if (kk >= T) continue;
      const size_t o = (rowb + kk) * (size_t)(a.Hkv * DH) + kvh * DH + (lane & 15);
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        base[(size_t)hh * plane + o + 16 * t] = dk[t][r];
        base[(size_t)(grp + hh) * plane + o + 16 * t] = dv[t][r];
      }
    }
    return;
  }
  const float scale = 1.0f / sqrtf((float)DH);
  const int half = DH / 2;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int kk = kw + 4 * (lane >> 4) + r;
    if (kk >= T) continue;
    bf16* dvr = a.dv + (rowb + kk) * a.ldk + kvh * DH;
    bf16* dkr = a.dk + (rowb + kk) * a.ldk + kvh * DH;
#pragma unroll
    for (int t = 0; t < NT / 2; ++t) {
      const int e = t * 16 + (lane & 15);
      const float2 cs = *(const float2*)(a.cs + 2 * ((size_t)kk * half + e));
      const float d1 = dk[t][r] * scale, d2 = dk[t + NT / 2][r] * scale;
      dkr[e] = to_bf16(d1 * cs.x + d2 * cs.y);
      dkr[e + half] = to_bf16(d2 * cs.x - d1 * cs.y);
      dvr[e] = to_bf16(dv[t][r]);
      dvr[e + half] = to_bf16(dv[t + NT / 2][r]);
    }
  }
}

// dQ for a block of 64 queries (4 waves of 16) of one head, key blocks of KB. With
// `nck` > 0 the key range is split into chunks of `ck` keys, one per workgroup
// (blockIdx.x = query tile * nck + chunk), each storing its fp32 partial dQ^T rows;
// k_attn_dq_reduce sums them in chunk order and finishes dQ (scale, RoPE backward).
//
// PF: the next key block is loaded into registers while the current one is multiplied.
// Without it (head dim 256) the kernel stays within 256 registers per lane, so that two
// workgroups share a compute unit and hide each other's load latency instead.
template <int DH, int KB, bool PF>
__global__ __launch_bounds__(256, PF ? 1 : 2) void k_attn_bwd_dq(const AttnArgs a, float* part, int nck, int ck) {
  constexpr int LDN = DH + 8, LDT_ = KB + 4, NKS = DH / 32, NT = DH / 16, NKT = KB / 16;
  __shared__ __attribute__((aligned(16))) u16 Ks[KB * LDN];   // fp16 (scores)
  __shared__ __attribute__((aligned(16))) u16 Vs[KB * LDN];   // bf16 (dP)
  __shared__ __attribute__((aligned(16))) u16 Kt[DH * LDT_];  // bf16 (dQ product)
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const TileId id = attn_tile(nck);
  const int tile = nck ? id.x / nck : id.x, chunk = nck ? id.x % nck : 0;
  const int T = a.T, h = id.y, b = id.z, grp = a.Hq / a.Hkv, kvh = h / grp;
  const int q0 = tile * 64, qw = q0 + 16 * w, q = qw + (lane & 15);
  const VisRange kvis = keys_of_query(q, a.T, a.window);
  const float sc = LOG2E / sqrtf((float)DH);
  const size_t rowb = (size_t)b * T;

  int kv_lo = 0;
  if (a.window) kv_lo = max(0, q0 - a.window + 1) & ~(KB - 1);
  int kv_hi = min(T, q0 + 64);
  if (nck) {
    kv_lo += chunk * ck;
    if (kv_lo >= kv_hi) return;  // the whole workgroup: no chunk here
    kv_hi = min(kv_hi, kv_lo + ck);
  }

  StageB<KB, DH, 256> kst;  // K: row-major fp16 (scores) and transposed bf16 (dQ product)
  StageN<KB, DH, 256> vst;  // V: row-major, converted to bf16
  const rsrc_t rK = seq_rsrc(a.k, rowb, T, a.ldk, kvh * DH, DH), rV = seq_rsrc(a.v, rowb, T, a.ldk, kvh * DH, DH);
  auto gload = [&](int kv0) {
    kst.load_rs(rK, kv0, a.ldk, tid);
    vst.load_rs(rV, kv0, a.ldk, tid);
  };
  if (PF) gload(kv_lo);

  uint4 qf[NKS], dof[NKS];  // Q fp16, dO bf16
#pragma unroll
  for (int ks = 0; ks < NKS; ++ks) {
    const size_t off = (rowb + q) * a.ldq + h * DH + 32 * ks + 8 * (lane >> 4);
    qf[ks] = load_frag_global(a.q + off, q < T);
    dof[ks] = load_frag_global(a.dO + off, q < T);
  }
  const size_t si = ((size_t)b * a.Hq + h) * T + q;
  const float lse2 = q < T ? a.lse[si] * LOG2E : 0.f;
  const float del = q < T ? a.delta[si] : 0.f;
  f32x4 dq[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) dq[t] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int kv0 = kv_lo; kv0 < kv_hi; kv0 += KB) {
    if (!PF) gload(kv0);
    __syncthreads();  // every wave is done with the previous block's tiles
    kst.template store_n<false>(Ks, LDN, tid);
    kst.template store_t<true>(Kt, LDT_, tid);
    vst.template store<true>(Vs, LDN, tid);
    __syncthreads();
    if (PF && kv0 + KB < kv_hi) gload(kv0 + KB);  // next block in flight during this one
    f32x4 s[NKT], dp[NKT];
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt) {
      s[kt] = f32x4{0.f, 0.f, 0.f, 0.f};
      dp[kt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks) {
        s[kt] = mfma16_raw<OpF16>(frag_rows(Ks, LDN, kt * 16, ks * 32, lane), qf[ks], s[kt]);
        dp[kt] = mfma16_raw<OpBF16>(frag_rows(Vs, LDN, kt * 16, ks * 32, lane), dof[ks], dp[kt]);
      }
    }
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const bool vis = visible(kvis, kv0 + kt * 16 + 4 * (lane >> 4) + r);
        const float p = vis ? exp2_fast(s[kt][r] * sc - lse2) : 0.f;
        dp[kt][r] = p * (dp[kt][r] - del);
      }
#pragma unroll
    for (int kp = 0; kp < NKT / 2; ++kp) {
      const uint4 df = pack_frag<OpBF16>(dp[2 * kp], dp[2 * kp + 1]);
#pragma unroll
      for (int t = 0; t < NT; ++t) dq[t] = mfma16_raw<OpBF16>(frag_perm(Kt, LDT_, t * 16, kp * 32, lane), df, dq[t]);
    }
  }
  if (q >= T) return;
  if (nck) {
    // chunk partial [chunk][B*T][Hq*DH], raw dQ^T sums (lane holds e = 16t + 4g + r)
    float* pr = part + ((size_t)chunk * a.B * T + rowb + q) * (size_t)(a.Hq * DH) + h * DH;
#pragma unroll
    for (int t = 0; t < NT; ++t)
      *(float4*)(pr + t * 16 + 4 * (lane >> 4)) = make_float4(dq[t][0], dq[t][1], dq[t][2], dq[t][3]);
    return;
  }
  {
    // lane holds dQ^T rows e = 16t + 4g + r of query q; pairs (e, e + dh/2) share the lane
    const float scale = 1.0f / sqrtf((float)DH);
    const int half = DH / 2;
    bf16* dqr = a.dq + (rowb + q) * a.ldq + h * DH;
#pragma unroll
    for (int t = 0; t < NT / 2; ++t) {
      float lo[4], hi[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int e = t * 16 + 4 * (lane >> 4) + r;
        const float2 cs = *(const float2*)(a.cs + 2 * ((size_t)q * half + e));
        const float d1 = dq[t][r] * scale, d2 = dq[t + NT / 2][r] * scale;
        lo[r] = d1 * cs.x + d2 * cs.y;
        hi[r] = d2 * cs.x - d1 * cs.y;
      }
      const int e0 = t * 16 + 4 * (lane >> 4);
      *(uint2*)(dqr + e0) = make_uint2(pack_bf16x2(lo[0], lo[1]), pack_bf16x2(lo[2], lo[3]));
      *(uint2*)(dqr + e0 + half) = make_uint2(pack_bf16x2(hi[0], hi[1]), pack_bf16x2(hi[2], hi[3]));
    }
  }
}

// Sum of the key-chunk partials of k_attn_bwd_dq in chunk order, scale 1/sqrt(dh), RoPE
// backward, bf16 store. One thread per (token, head, 4 columns of the first half of the
// head) and their partners e + dh/2.
__global__ void k_attn_dq_reduce(const AttnArgs a, const float* part, int nck, int ck, int KB) {
  const int half = a.dh / 2, q4 = half / 4;
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (size_t)a.B * a.T * a.Hq * q4) return;
  const int e = (int)(i % q4) * 4;
  const int h = (int)((i / q4) % a.Hq);
  const size_t row = i / ((size_t)q4 * a.Hq);
  const int t = (int)(row % a.T);
  const int n = fwd_tile_chunks(t / 64, a.T, a.window, KB, ck);
  const size_t ldp = (size_t)a.Hq * a.dh, plane = (size_t)a.B * a.T * ldp;
  const float* p0 = part + row * ldp + h * a.dh + e;
  float d1[4] = {0, 0, 0, 0}, d2[4] = {0, 0, 0, 0};
  for (int c = 0; c < n; ++c) {
    const float4 x = *(const float4*)(p0 + c * plane), y = *(const float4*)(p0 + c * plane + half);
    d1[0] += x.x; d1[1] += x.y; d1[2] += x.z; d1[3] += x.w;
    d2[0] += y.x; d2[1] += y.y; d2[2] += y.z; d2[3] += y.w;
  }
  const float scale = 1.0f / sqrtf((float)a.dh);
  float lo[4], hi[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const float2 cs = *(const float2*)(a.cs + 2 * ((size_t)t * half + e + j));
    const float u = d1[j] * scale, v = d2[j] * scale;
    lo[j] = u * cs.x + v * cs.y;
    hi[j] = v * cs.x - u * cs.y;
  }
  bf16* dqr = a.dq + row * a.ldq + h * a.dh + e;
  *(uint2*)dqr = make_uint2(pack_bf16x2(lo[0], lo[1]), pack_bf16x2(lo[2], lo[3]));
  *(uint2*)(dqr + half) = make_uint2(pack_bf16x2(hi[0], hi[1]), pack_bf16x2(hi[2], hi[3]));
}


// dK, dV with 32-key waves (v_mfma_f32_32x32x16). Each wave keeps its 32 keys' K (fp16)
// and V (bf16) as B operands in registers and its dK^T, dV^T accumulators for all head
// dims; the workgroup walks the query tiles (32 queries) that can see its keys. Per tile:
// S = Q K^T and dP = dO V^T put one key per lane column and 16 queries in its registers
// (queries 8(r/4) + 4h + r%4), P = exp(S - lse) and dS = P (dP - delta) read the row
// statistics from LDS, and dV^T += dO^T P, dK^T += Q^T dS take P, dS straight from
// registers as B operands (queries {4h..4h+3, 8+4h..8+4h+3} of a 16-query step) with the
// dO^T / Q^T fragments read in the same query order. Q and dO are staged row-major (Q
// fp16 for the scores, dO bf16) and transposed (bf16) from 8x8 register blocks; the next
// tile is loaded into registers while the current one is multiplied. With grouped-query
// attention every query head stores fp32 partials that k_attn_dkdv_reduce sums in head
// order; otherwise the epilogue scales dK, applies the RoPE backward and stores bf16.
template <int DH, int NW>
__global__ __launch_bounds__(64 * NW) void k_attn_bwd_kv32(const AttnArgs a, float* part) {
  constexpr int NTH = 64 * NW, QB = 32, LDN = DH + 8, LDT = QB + 8;
  constexpr int NKS = DH / 16, NTO = DH / 32;
  constexpr int NBT = (QB / 8) * (DH / 8);   // 8x8 blocks per tensor (Q, dO) and tile
  constexpr int BPT = (2 * NBT + NTH - 1) / NTH;
  __shared__ __attribute__((aligned(16))) u16 Qs[QB * LDN];   // fp16 [q][e]
  __shared__ __attribute__((aligned(16))) u16 dOs[QB * LDN];  // bf16 [q][e]
  __shared__ __attribute__((aligned(16))) u16 Qt[DH * LDT];   // bf16 [e][q]
  __shared__ __attribute__((aligned(16))) u16 dOt[DH * LDT];  // bf16 [e][q]
  __shared__ __attribute__((aligned(16))) float lse_s[QB], del_s[QB];
  const int tid = threadIdx.x, lane = tid & 63, w = __builtin_amdgcn_readfirstlane(tid >> 6), hl = lane >> 5;
  const TileId id = attn_tile(0);
  const int T = a.T, h = id.y, b = id.z, grp = a.Hq / a.Hkv, kvh = h / grp, hh = h % grp;
  const int k0 = id.x * (32 * NW), kw = k0 + 32 * w, key = kw + (lane & 31);
  const VisRange qvis = queries_of_key(key, T, a.window);
  const float sc = LOG2E / sqrtf((float)DH);
  const size_t rowb = (size_t)b * T;

  uint4 kf[NKS], vf[NKS];
#pragma unroll
  for (int ks = 0; ks < NKS; ++ks) {
    const size_t off = (rowb + key) * a.ldk + kvh * DH + 16 * ks + 8 * hl;
    kf[ks] = load_frag_global(a.k + off, key < T);
    vf[ks] = f16x8_to_bf16x8(load_frag_global(a.v + off, key < T));
  }
  f32x16 dk[NTO], dv[NTO];
#pragma unroll
  for (int t = 0; t < NTO; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) dk[t][r] = dv[t][r] = 0.f;

  const int q_lo = k0 & ~(QB - 1);
  const int q_hi = a.window ? min(T, k0 + 32 * NW - 1 + a.window) : T;

  uint4 br[BPT][8];
  float st_lse = 0.f, st_del = 0.f;
  const size_t stat0 = ((size_t)b * a.Hq + h) * T;  // this (sequence, head)'s row statistics
  const rsrc_t rL = make_rsrc(a.lse + stat0, (size_t)T * 4), rD = make_rsrc(a.delta + stat0, (size_t)T * 4);
  // Q and dO rows of this sequence and head through buffer resources (rows past T read as
  // zero); per-lane offsets fixed for the kernel, wave-uniform row offsets
  const rsrc_t rQ = seq_rsrc(a.q, rowb, T, a.ldq, h * DH, DH), rdO = seq_rsrc(a.dO, rowb, T, a.ldq, h * DH, DH);
  uint32_t boff[BPT];
#pragma unroll
  for (int i = 0; i < BPT; ++i) {
    const int bl = min(tid + NTH * i, 2 * NBT - 1), lb = bl % NBT, rb = lb % (QB / 8), cb = lb / (QB / 8);
    boff[i] = (uint32_t)(((rb * 8) * a.ldq + cb * 8) * 2);
  }
  const uint32_t rowB = (uint32_t)a.ldq * 2;
  auto gload = [&](int qb0) {
#pragma unroll
    for (int i = 0; i < BPT; ++i) {
      // wave-uniform (NBT is a multiple of 64): the resource stays in scalar registers
      const bool q_tens = min(__builtin_amdgcn_readfirstlane(tid) + NTH * i, 2 * NBT - 1) < NBT;
#pragma unroll
      for (int j = 0; j < 8; ++j)
        br[i][j] = bload128s(q_tens ? rQ : rdO, boff[i], (uint32_t)(qb0 + j) * rowB);
    }
    // the row statistics of queries qb0 + tid (tid < QB) through buffer loads, without a
    // branch, and scaled only when stored: a use right after the load would make the wave wait
    // for it, and so for every tile load issued before it
    {
      const int qq = qb0 + tid;
      const uint32_t so = (tid < QB && qq < T) ? (uint32_t)qq * 4 : 0x80000000u;
      st_lse = __uint_as_float(bload32(rL, so));
      st_del = __uint_as_float(bload32(rD, so));
    }
  };
  auto sstore = [&]() {
#pragma unroll
    for (int i = 0; i < BPT; ++i) {
      const int bl = tid + NTH * i, tens = bl / NBT, lb = bl % NBT, rb = lb % (QB / 8), cb = lb / (QB / 8);
      if (bl >= 2 * NBT) continue;
      u16* nrm = tens == 0 ? Qs : dOs;
      u16* trn = tens == 0 ? Qt : dOt;
      uint32_t in[8][4];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        *(uint4*)(nrm + (rb * 8 + j) * LDN + cb * 8) = br[i][j];
        const uint4 v = tens == 0 ? f16x8_to_bf16x8(br[i][j]) : br[i][j];
        in[j][0] = v.x; in[j][1] = v.y; in[j][2] = v.z; in[j][3] = v.w;
      }
#pragma unroll
      for (int jc = 0; jc < 8; ++jc) {
        const int d = jc >> 1;
        uint4 o;
        if (jc & 1) {
          o = make_uint4(perm_hi16(in[0][d], in[1][d]), perm_hi16(in[2][d], in[3][d]), perm_hi16(in[4][d], in[5][d]),
                         perm_hi16(in[6][d], in[7][d]));
        } else {
          o = make_uint4(perm_lo16(in[0][d], in[1][d]), perm_lo16(in[2][d], in[3][d]), perm_lo16(in[4][d], in[5][d]),
                         perm_lo16(in[6][d], in[7][d]));
        }
        *(uint4*)(trn + (cb * 8 + jc) * LDT + rb * 8) = o;
      }
    }
    if (tid < QB) {
      lse_s[tid] = st_lse * LOG2E;
      del_s[tid] = st_del;
    }
  };

  if (q_lo < q_hi) gload(q_lo);
  for (int qb0 = q_lo; qb0 < q_hi; qb0 += QB) {
    __syncthreads();  // every wave is done with the previous tile
    sstore();
    __syncthreads();
    // next tile in flight during this one; issued after the last tile too (rows past T read as
    // zero, rows past the range are unused), since loads behind a branch leave the compiler
    // only a full wait for them before the next MFMA
    gload(qb0 + QB);
    // nothing visible for this wave: all queries before its keys, or past its window
    if (qb0 + QB - 1 < kw || (a.window && qb0 > kw + 31 + a.window - 1)) continue;
    f32x16 sv, dp;
#pragma unroll
    for (int r = 0; r < 16; ++r) sv[r] = dp[r] = 0.f;
    {
      const u16* qp = Qs + (lane & 31) * LDN + 8 * hl;
      const u16* op = dOs + (lane & 31) * LDN + 8 * hl;
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks) {
        sv = mfma32_f16(*(const uint4*)(qp + 16 * ks), kf[ks], sv);
        dp = mfma32_bf16(*(const uint4*)(op + 16 * ks), vf[ks], dp);
      }
    }
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const float4 l4 = *(const float4*)(lse_s + 8 * g + 4 * hl), d4 = *(const float4*)(del_s + 8 * g + 4 * hl);
      const float lv[4] = {l4.x, l4.y, l4.z, l4.w}, dl[4] = {d4.x, d4.y, d4.z, d4.w};
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        const int r = 4 * g + rr;
        const bool vis = visible(qvis, qb0 + 8 * g + 4 * hl + rr);
        const float p = vis ? exp2_fast(sv[r] * sc - lv[rr]) : 0.f;
        sv[r] = p;
        dp[r] = p * (dp[r] - dl[rr]);
      }
    }
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      const int r0 = 8 * kk;
      const uint4 pf = make_uint4(pack_bf16x2(sv[r0 + 0], sv[r0 + 1]), pack_bf16x2(sv[r0 + 2], sv[r0 + 3]),
                                  pack_bf16x2(sv[r0 + 4], sv[r0 + 5]), pack_bf16x2(sv[r0 + 6], sv[r0 + 7]));
      const uint4 df = make_uint4(pack_bf16x2(dp[r0 + 0], dp[r0 + 1]), pack_bf16x2(dp[r0 + 2], dp[r0 + 3]),
                                  pack_bf16x2(dp[r0 + 4], dp[r0 + 5]), pack_bf16x2(dp[r0 + 6], dp[r0 + 7]));
#pragma unroll
      for (int t = 0; t < NTO; ++t) {
        const int rowoff = (t * 32 + (lane & 31)) * LDT + kk * 16 + 4 * hl;
        const uint2 o0 = *(const uint2*)(dOt + rowoff), o1 = *(const uint2*)(dOt + rowoff + 8);
        dv[t] = mfma32_bf16(make_uint4(o0.x, o0.y, o1.x, o1.y), pf, dv[t]);
        const uint2 q0v = *(const uint2*)(Qt + rowoff), q1v = *(const uint2*)(Qt + rowoff + 8);
        dk[t] = mfma32_bf16(make_uint4(q0v.x, q0v.y, q1v.x, q1v.y), df, dk[t]);
      }
    }
  }
  if (key >= T) return;
  // lane holds dK^T, dV^T rows e = 32t + 8g + 4h + rr of key `key`
  if (grp > 1) {
    const size_t plane = (size_t)a.B * T * a.Hkv * DH;
    const size_t o = (rowb + key) * (size_t)(a.Hkv * DH) + kvh * DH;
#pragma unroll
    for (int t = 0; t < NTO; ++t)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int e0 = 32 * t + 8 * g + 4 * hl;
        *(float4*)(part + (size_t)hh * plane + o + e0) =
            make_float4(dk[t][4 * g], dk[t][4 * g + 1], dk[t][4 * g + 2], dk[t][4 * g + 3]);
        *(float4*)(part + (size_t)(grp + hh) * plane + o + e0) =
            make_float4(dv[t][4 * g], dv[t][4 * g + 1], dv[t][4 * g + 2], dv[t][4 * g + 3]);
      }
    return;
  }
  const float scale = 1.0f / sqrtf((float)DH);
  constexpr int half = DH / 2;
  bf16* dvr = a.dv + (rowb + key) * a.ldk + kvh * DH;
  bf16* dkr = a.dk + (rowb + key) * a.ldk + kvh * DH;
#pragma unroll
  for (int t = 0; t < NTO / 2; ++t)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int e0 = 32 * t + 8 * g + 4 * hl;
      float lo[4], hi[4];
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        const float2 cs = *(const float2*)(a.cs + 2 * ((size_t)key * half + e0 + rr));
        const float d1 = dk[t][4 * g + rr] * scale, d2 = dk[t + NTO / 2][4 * g + rr] * scale;
        lo[rr] = d1 * cs.x + d2 * cs.y;
        hi[rr] = d2 * cs.x - d1 * cs.y;
      }
      *(uint2*)(dkr + e0) = make_uint2(pack_bf16x2(lo[0], lo[1]), pack_bf16x2(lo[2], lo[3]));
      *(uint2*)(dkr + e0 + half) = make_uint2(pack_bf16x2(hi[0], hi[1]), pack_bf16x2(hi[2], hi[3]));
      *(uint2*)(dvr + e0) = make_uint2(pack_bf16x2(dv[t][4 * g], dv[t][4 * g + 1]), pack_bf16x2(dv[t][4 * g + 2], dv[t][4 * g + 3]));
      *(uint2*)(dvr + e0 + half) = make_uint2(pack_bf16x2(dv[t + NTO / 2][4 * g], dv[t + NTO / 2][4 * g + 1]),
                                              pack_bf16x2(dv[t + NTO / 2][4 * g + 2], dv[t + NTO / 2][4 * g + 3]));
    }
}


// dK, dV at head dim 256 with 32-key wave pairs (v_mfma_f32_32x32x16). The 32-key kernel
// above would need K, V (128 registers) and dK^T, dV^T (256 accumulators) in every wave;
// here the two waves of a pair share those 32 keys: the first keeps K and accumulates
// dV^T, the second keeps V and accumulates dK^T. Per query tile (32 queries, staged as in
// k_attn_bwd_kv32): the first wave computes S = Q K^T and P = exp(S - lse), hands P to its
// partner through LDS (fp32, one 16-value slot per lane: the partner's dP tile has the same
// lane layout) and adds dO^T P into dV^T; the second computes dP = dO V^T, then dS = P (dP -
// delta) and adds Q^T dS into dK^T. Each wave thus holds 64 operand registers and 128
// accumulators, and every Q / dO fragment read from LDS feeds a 32-key MFMA.
template <int NP>
__global__ __launch_bounds__(128 * NP) void k_attn_bwd_kv32p(const AttnArgs a, float* part) {
  constexpr int DH = 256, NTH = 128 * NP, QB = 32, LDN = DH + 8, LDT = QB + 8;
  constexpr int NKS = DH / 16, NTO = DH / 32;
  constexpr int NBT = (QB / 8) * (DH / 8);   // 8x8 blocks per tensor (Q, dO) and tile
  constexpr int BPT = (2 * NBT + NTH - 1) / NTH;
  __shared__ __attribute__((aligned(16))) u16 Qs[QB * LDN];   // fp16 [q][e]
  __shared__ __attribute__((aligned(16))) u16 dOs[QB * LDN];  // bf16 [q][e]
  __shared__ __attribute__((aligned(16))) u16 Qt[DH * LDT];   // bf16 [e][q]
  __shared__ __attribute__((aligned(16))) u16 dOt[DH * LDT];  // bf16 [e][q]
  __shared__ __attribute__((aligned(16))) float Ps[NP][16][64];  // P of each pair, [r][lane]
  __shared__ __attribute__((aligned(16))) float lse_s[QB], del_s[QB];
  const int tid = threadIdx.x, lane = tid & 63, w = __builtin_amdgcn_readfirstlane(tid >> 6), hl = lane >> 5;
  const int pair = w >> 1, role = w & 1;  // role 0: K, P, dV; role 1: V, dP, dS, dK
  const TileId id = attn_tile(0);
  const int T = a.T, h = id.y, b = id.z, grp = a.Hq / a.Hkv, kvh = h / grp, hh = h % grp;
  const int k0 = id.x * (32 * NP), kw = k0 + 32 * pair, key = kw + (lane & 31);
  const VisRange qvis = queries_of_key(key, T, a.window);
  const float sc = LOG2E / sqrtf((float)DH);
  const size_t rowb = (size_t)b * T;

  uint4 kv[NKS];  // K (fp16) or V (bf16) of the pair's keys
#pragma unroll
  for (int ks = 0; ks < NKS; ++ks) {
    const size_t off = (rowb + key) * a.ldk + kvh * DH + 16 * ks + 8 * hl;
    const uint4 x = load_frag_global((role == 0 ? a.k : a.v) + off, key < T);
    kv[ks] = role == 0 ? x : f16x8_to_bf16x8(x);
  }
  f32x16 acc[NTO];  // dV^T (role 0) or dK^T (role 1)
#pragma unroll
  for (int t = 0; t < NTO; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[t][r] = 0.f;

  const int q_lo = k0 & ~(QB - 1);
  const int q_hi = a.window ? min(T, k0 + 32 * NP - 1 + a.window) : T;

  uint4 br[BPT][8];
  float st_lse = 0.f, st_del = 0.f;
  const size_t stat0 = ((size_t)b * a.Hq + h) * T;  // this (sequence, head)'s row statistics
  const rsrc_t rL = make_rsrc(a.lse + stat0, (size_t)T * 4), rD = make_rsrc(a.delta + stat0, (size_t)T * 4);
  // Q and dO rows of this sequence and head through buffer resources (rows past T read as
  // zero); per-lane offsets fixed for the kernel, wave-uniform row offsets
  const rsrc_t rQ = seq_rsrc(a.q, rowb, T, a.ldq, h * DH, DH), rdO = seq_rsrc(a.dO, rowb, T, a.ldq, h * DH, DH);
  uint32_t boff[BPT];
#pragma unroll
  for (int i = 0; i < BPT; ++i) {
    const int bl = min(tid + NTH * i, 2 * NBT - 1), lb = bl % NBT, rb = lb % (QB / 8), cb = lb / (QB / 8);
    boff[i] = (uint32_t)(((rb * 8) * a.ldq + cb * 8) * 2);
  }
  const uint32_t rowB = (uint32_t)a.ldq * 2;
  auto gload = [&](int qb0) {
#pragma unroll
    for (int i = 0; i < BPT; ++i) {
      // wave-uniform (NBT is a multiple of 64): the resource stays in scalar registers
      const bool q_tens = min(__builtin_amdgcn_readfirstlane(tid) + NTH * i, 2 * NBT - 1) < NBT;
#pragma unroll
      for (int j = 0; j < 8; ++j)
        br[i][j] = bload128s(q_tens ? rQ : rdO, boff[i], (uint32_t)(qb0 + j) * rowB);
    }
    // the row statistics of queries qb0 + tid (tid < QB) through buffer loads, without a
    // branch, and scaled only when stored: a use right after the load would make the wave wait
    // for it, and so for every tile load issued before it
    {
      const int qq = qb0 + tid;
      const uint32_t so = (tid < QB && qq < T) ? (uint32_t)qq * 4 : 0x80000000u;
      st_lse = __uint_as_float(bload32(rL, so));
      st_del = __uint_as_float(bload32(rD, so));
    }
  };
  auto sstore = [&]() {
#pragma unroll
    for (int i = 0; i < BPT; ++i) {
      const int bl = tid + NTH * i, tens = bl / NBT, lb = bl % NBT, rb = lb % (QB / 8), cb = lb / (QB / 8);
      if (bl >= 2 * NBT) continue;
      u16* nrm = tens == 0 ? Qs : dOs;
      u16* trn = tens == 0 ? Qt : dOt;
      uint32_t in[8][4];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        *(uint4*)(nrm + (rb * 8 + j) * LDN + cb * 8) = br[i][j];
        const uint4 v = tens == 0 ? f16x8_to_bf16x8(br[i][j]) : br[i][j];
        in[j][0] = v.x; in[j][1] = v.y; in[j][2] = v.z; in[j][3] = v.w;
      }
#pragma unroll
      for (int jc = 0; jc < 8; ++jc) {
        const int d = jc >> 1;
        uint4 o;
        if (jc & 1) {
          o = make_uint4(perm_hi16(in[0][d], in[1][d]), perm_hi16(in[2][d], in[3][d]), perm_hi16(in[4][d], in[5][d]),
                         perm_hi16(in[6][d], in[7][d]));
        } else {
          o = make_uint4(perm_lo16(in[0][d], in[1][d]), perm_lo16(in[2][d], in[3][d]), perm_lo16(in[4][d], in[5][d]),
                         perm_lo16(in[6][d], in[7][d]));
        }
        *(uint4*)(trn + (cb * 8 + jc) * LDT + rb * 8) = o;
      }
    }
    if (tid < QB) {
      lse_s[tid] = st_lse * LOG2E;
      del_s[tid] = st_del;
    }
  };

  if (q_lo < q_hi) gload(q_lo);
  for (int qb0 = q_lo; qb0 < q_hi; qb0 += QB) {
    __syncthreads();  // every wave is done with the previous tile (and its P slot)
    sstore();
    __syncthreads();
    // next tile in flight during this one; issued after the last tile too (rows past T read as
    // zero, rows past the range are unused), since loads behind a branch leave the compiler
    // only a full wait for them before the next MFMA
    gload(qb0 + QB);
    // A pair with nothing visible in this tile (all its queries before its keys, or past its
    // window) runs the MFMAs anyway: its P and dS are masked to zero, so they add nothing.
    // Without a branch around them the accumulators stay in the accumulator registers across
    // tiles (with one, the compiler copied all 128 out and back on every tile).
    f32x16 x;  // S then P (role 0), dP then dS (role 1)
#pragma unroll
    for (int r = 0; r < 16; ++r) x[r] = 0.f;
    {
      const u16* src = (role == 0 ? Qs : dOs) + (lane & 31) * LDN + 8 * hl;
      if (role == 0) {
        x = lds_chain<3>(src, kv, x, [](uint4 p, uint4 q, f32x16 c) { return mfma32_f16(p, q, c); });
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const float4 l4 = *(const float4*)(lse_s + 8 * g + 4 * hl);
          const float lv[4] = {l4.x, l4.y, l4.z, l4.w};
#pragma unroll
          for (int rr = 0; rr < 4; ++rr) {
            const int r = 4 * g + rr;
            const bool vis = visible(qvis, qb0 + 8 * g + 4 * hl + rr);
            x[r] = vis ? exp2_fast(x[r] * sc - lv[rr]) : 0.f;
            Ps[pair][r][lane] = x[r];
          }
        }
      } else {
        x = lds_chain<3>(src, kv, x, [](uint4 p, uint4 q, f32x16 c) { return mfma32_bf16(p, q, c); });
      }
    }
    __syncthreads();  // P of every pair is in LDS
    {
      if (role == 1) {
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const float4 d4 = *(const float4*)(del_s + 8 * g + 4 * hl);
          const float dl[4] = {d4.x, d4.y, d4.z, d4.w};
#pragma unroll
          for (int rr = 0; rr < 4; ++rr) {
            const int r = 4 * g + rr;
            x[r] = Ps[pair][r][lane] * (x[r] - dl[rr]);
          }
        }
      }
      const u16* opnd = role == 0 ? dOt : Qt;
      uint4 f[2];
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
        const int r0 = 8 * kk;
        f[kk] = make_uint4(pack_bf16x2(x[r0 + 0], x[r0 + 1]), pack_bf16x2(x[r0 + 2], x[r0 + 3]),
                           pack_bf16x2(x[r0 + 4], x[r0 + 5]), pack_bf16x2(x[r0 + 6], x[r0 + 7]));
      }
      // 2 x NTO MFMAs in (key step, output tile) order, operand fragments read three ahead
      constexpr int FA = 3, NM = 2 * NTO;
      uint4 ob[FA + 2];
      auto rdo = [&](int i) {
        const int rowoff = ((i % NTO) * 32 + (lane & 31)) * LDT + (i / NTO) * 16 + 4 * hl;
        const uint2 o0 = *(const uint2*)(opnd + rowoff), o1 = *(const uint2*)(opnd + rowoff + 8);
        return make_uint4(o0.x, o0.y, o1.x, o1.y);
      };
#pragma unroll
      for (int i = 0; i < FA; ++i) ob[i] = rdo(i);
#pragma unroll
      for (int i = 0; i < NM; ++i) {
        if (i + FA < NM) ob[(i + FA) % (FA + 2)] = rdo(i + FA);
        acc[i % NTO] = mfma32_bf16(ob[i % (FA + 2)], f[i / NTO], acc[i % NTO]);
      }
      __builtin_amdgcn_sched_group_barrier(0x100, FA, 0);
#pragma unroll
      for (int i = 0; i < NM; ++i) {
        if (i + FA < NM) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      }
    }
  }
  if (key >= T) return;
  // lane holds dK^T or dV^T rows e = 32t + 8g + 4h + rr of key `key`
  if (grp > 1) {
    const size_t plane = (size_t)a.B * T * a.Hkv * DH;
    const size_t o = (rowb + key) * (size_t)(a.Hkv * DH) + kvh * DH;
    float* dst = part + (size_t)(role == 0 ? grp + hh : hh) * plane + o;
#pragma unroll
    for (int t = 0; t < NTO; ++t)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int e0 = 32 * t + 8 * g + 4 * hl;
        *(float4*)(dst + e0) = make_float4(acc[t][4 * g], acc[t][4 * g + 1], acc[t][4 * g + 2], acc[t][4 * g + 3]);
      }
    return;
  }
  constexpr int half = DH / 2;
  if (role == 0) {
    bf16* dvr = a.dv + (rowb + key) * a.ldk + kvh * DH;
#pragma unroll
    for (int t = 0; t < NTO; ++t)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int e0 = 32 * t + 8 * g + 4 * hl;
        *(uint2*)(dvr + e0) =
            make_uint2(pack_bf16x2(acc[t][4 * g], acc[t][4 * g + 1]), pack_bf16x2(acc[t][4 * g + 2], acc[t][4 * g + 3]));
      }
    return;
  }
  const float scale = 1.0f / sqrtf((float)DH);
  bf16* dkr = a.dk + (rowb + key) * a.ldk + kvh * DH;
#pragma unroll
  for (int t = 0; t < NTO / 2; ++t)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int e0 = 32 * t + 8 * g + 4 * hl;
      float lo[4], hi[4];
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        const float2 cs = *(const float2*)(a.cs + 2 * ((size_t)key * half + e0 + rr));
        const float d1 = acc[t][4 * g + rr] * scale, d2 = acc[t + NTO / 2][4 * g + rr] * scale;
        lo[rr] = d1 * cs.x + d2 * cs.y;
        hi[rr] = d2 * cs.x - d1 * cs.y;
      }
      *(uint2*)(dkr + e0) = make_uint2(pack_bf16x2(lo[0], lo[1]), pack_bf16x2(lo[2], lo[3]));
      *(uint2*)(dkr + e0 + half) = make_uint2(pack_bf16x2(hi[0], hi[1]), pack_bf16x2(hi[2], hi[3]));
    }
}

// Number of query chunks of `cq` queries that key block `kblk` (64 keys) of
// k_attn_bwd_dkdv visits.
__host__ __device__ inline int kv_block_chunks(int kblk, int T, int window, int cq) {
  const int k0 = kblk * 64;
  const int hi = window ? (T < k0 + 64 + window - 1 ? T : k0 + 64 + window - 1) : T;
  return hi > k0 ? (hi - k0 + cq - 1) / cq : 0;
}

// dK/dV from the partial planes of the key-block kernels: sum the query chunks (nck > 0;
// else one) and, within each, the query heads of the KV group, in that order; scale dK by
// 1/sqrt(dh), rotate it back (RoPE backward), store bf16. One thread per (token, kv
// head, 4 columns of the first half of the head) and their partners.
__global__ void k_attn_dkdv_reduce(const AttnArgs a, const float* part, int nck, int cq) {
  const int half = a.dh / 2, q4 = half / 4;
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const size_t total = (size_t)a.B * a.T * a.Hkv * q4;
  if (i >= total) return;
  const int e = (int)(i % q4) * 4;
  const int kvh = (int)((i / q4) % a.Hkv);
  const size_t row = i / ((size_t)q4 * a.Hkv);
  const int t = (int)(row % a.T), grp = a.Hq / a.Hkv;
  const int n = nck ? kv_block_chunks(t / 64, a.T, a.window, cq) : 1;
  const size_t plane = (size_t)a.B * a.T * a.Hkv * a.dh;
  const size_t o = row * (size_t)(a.Hkv * a.dh) + kvh * a.dh + e;
  float k1[4] = {0, 0, 0, 0}, k2[4] = {0, 0, 0, 0}, v1[4] = {0, 0, 0, 0}, v2[4] = {0, 0, 0, 0};
  for (int c = 0; c < n; ++c) {
    const float* base = part + (size_t)c * 2 * grp * plane;
    for (int g = 0; g < grp; ++g) {
      const float4 a1 = *(const float4*)(base + g * plane + o), a2 = *(const float4*)(base + g * plane + o + half);
      const float4 b1 = *(const float4*)(base + (grp + g) * plane + o);
      const float4 b2 = *(const float4*)(base + (grp + g) * plane + o + half);
      k1[0] += a1.x; k1[1] += a1.y; k1[2] += a1.z; k1[3] += a1.w;
      k2[0] += a2.x; k2[1] += a2.y; k2[2] += a2.z; k2[3] += a2.w;
      v1[0] += b1.x; v1[1] += b1.y; v1[2] += b1.z; v1[3] += b1.w;
      v2[0] += b2.x; v2[1] += b2.y; v2[2] += b2.z; v2[3] += b2.w;
    }
  }
  const float scale = 1.0f / sqrtf((float)a.dh);
  float lo[4], hi[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const float2 cs = *(const float2*)(a.cs + 2 * ((size_t)t * half + e + j));
    const float d1 = k1[j] * scale, d2 = k2[j] * scale;
    lo[j] = d1 * cs.x + d2 * cs.y;
    hi[j] = d2 * cs.x - d1 * cs.y;
  }
  *(uint2*)(a.dk + o) = make_uint2(pack_bf16x2(lo[0], lo[1]), pack_bf16x2(lo[2], lo[3]));
  *(uint2*)(a.dk + o + half) = make_uint2(pack_bf16x2(hi[0], hi[1]), pack_bf16x2(hi[2], hi[3]));
  *(uint2*)(a.dv + o) = make_uint2(pack_bf16x2(v1[0], v1[1]), pack_bf16x2(v1[2], v1[3]));
  *(uint2*)(a.dv + o + half) = make_uint2(pack_bf16x2(v2[0], v2[1]), pack_bf16x2(v2[2], v2[3]));
}

}  // namespace

// visible (query, key) pairs of one sequence and head
double visible_pairs(int T, int W) {
  double p = 0;
  for (int i = 0; i < T; ++i) p += (W && W < i + 1) ? W : i + 1;
  return p;
}

namespace {
int env_int(const char* name, int dflt) {
  const char* e = getenv(name);
  return e && *e ? atoi(e) : dflt;
}
}  // namespace

// Launch plan of the attention kernels for one shape. Short sequences with few heads give
// fewer 64-query (64-key) tiles than the chip has compute units, and each tile's loop over
// the other axis is a serial chain; there the loop is split into chunks, one workgroup
// each, and a merge kernel combines the chunks in a fixed order.
AttnPlan attn_plan(int B, int T, int Hq, int Hkv, int dh, int window) {
  // chunk lengths are whole 64-row tiles (multiples of every kernel's block)
  static const int use32 = env_int("MEBP_ATTN32", 1), split_on = env_int("MEBP_ATTN_SPLIT", 1),
                   CK = std::max(64, env_int("MEBP_ATTN_CK", 64) & ~63),
                   CQ = std::max(64, env_int("MEBP_ATTN_CQ", 128) & ~63);
  AttnPlan p{};
  const int nt64 = (T + 63) / 64;
  const size_t units64 = (size_t)nt64 * Hq * B;
  p.fwd32 = use32 && (size_t)((T + 127) / 128) * Hq * B >= 256;
  const bool split = split_on && units64 < 256 && nt64 > 1;
  if (split && !p.fwd32) {
    p.f_ck = CK;
    for (int t = 0; t < nt64; ++t) p.f_nck = std::max(p.f_nck, fwd_tile_chunks(t, T, window, 64, CK));
    // a chain of up to four key blocks costs less than the extra merge kernel
    if (p.f_nck <= 4) p.f_nck = 0;
  }
  if (split) {
    p.q_ck = CK;
    for (int t = 0; t < nt64; ++t) p.q_nck = std::max(p.q_nck, fwd_tile_chunks(t, T, window, dh == 256 ? 32 : 64, CK));
    if (p.q_nck <= 1) p.q_nck = 0;
  }
  if (split && dh != 128) {
    p.kv_cq = CQ;
    for (int k = 0; k < nt64; ++k) p.kv_nck = std::max(p.kv_nck, kv_block_chunks(k, T, window, CQ));
    if (p.kv_nck <= 1) p.kv_nck = 0;
  }
  const size_t rows = (size_t)B * T * Hq;
  p.fwd_floats = p.f_nck ? (size_t)p.f_nck * rows * (dh + 2) : 0;
  p.kv_floats = (p.kv_nck || Hq > Hkv) ? (size_t)std::max(p.kv_nck, 1) * 2 * rows * dh : 0;
  p.q_floats = p.q_nck ? (size_t)p.q_nck * rows * dh : 0;
  return p;
}

size_t attn_part_floats(int B, int T, int Hq, int Hkv, int dh, int window) {
  const AttnPlan p = attn_plan(B, T, Hq, Hkv, dh, window);
  return std::max(p.fwd_floats, p.kv_floats + p.q_floats);
}

hipError_t launch_attn_fwd(const AttnArgs& a, const SplitScratch& sc, hipStream_t st) {
  const double pairs = visible_pairs(a.T, a.window) * a.Hq * a.B;
  const double flops = 4.0 * a.dh * pairs;
  const double bytes = (double)a.B * a.T * (2.0 * a.Hq * a.dh * 2 + 2.0 * a.Hkv * a.dh * 2 + a.Hq * 4);
  const AttnPlan p = attn_plan(a.B, a.T, a.Hq, a.Hkv, a.dh, a.window);
  // (the kernels address a sequence's rows with 32-bit buffer offsets)
  if ((double)a.T * (a.ldq > a.ldk ? a.ldq : a.ldk) * 2 >= 2147483648.0) return hipErrorInvalidValue;
  if (p.fwd32) {
    // 128 queries per workgroup (4 waves of 32) when that still fills the chip
    const dim3 g2((a.T + 127) / 128, a.Hq, a.B);
#define FWD32(D) \
  MEBP_TIMED(st, "attn_fwd", flops, bytes, hipLaunchKernelGGL((k_attn_fwd32<D, 4>), g2, dim3(256), 0, st, a))
    switch (a.dh) {
      case 64: FWD32(64); break;
      case 128: FWD32(128); break;
      case 256: FWD32(256); break;
      default: return hipErrorInvalidValue;
    }
#undef FWD32
    return hipGetLastError();
  }
  if (p.f_nck && (!sc.part || sc.part_floats < p.fwd_floats)) return hipErrorInvalidValue;
  const dim3 grid(((a.T + 63) / 64) * (p.f_nck ? p.f_nck : 1), a.Hq, a.B);
#define FWD(D) \
  MEBP_TIMED(st, "attn_fwd", flops, bytes, hipLaunchKernelGGL(k_attn_fwd<D>, grid, dim3(256), 0, st, a, sc.part, p.f_nck, p.f_ck))
  switch (a.dh) {
    case 64: FWD(64); break;
    case 128: FWD(128); break;
    case 256: FWD(256); break;
    default: return hipErrorInvalidValue;
  }
#undef FWD
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !p.f_nck) return e;
  const size_t nc = (size_t)a.B * a.Hq * a.T * (a.dh / 8);
  const dim3 gc((unsigned)((nc + 255) / 256));
  const double cb = (double)p.fwd_floats * 4 + (double)a.B * a.T * a.Hq * (a.dh * 2 + 4);
#define CMB(D) \
  MEBP_TIMED(st, "attn_fwd_combine", 0.0, cb, hipLaunchKernelGGL(k_attn_fwd_combine<D>, gc, dim3(256), 0, st, a, (const float*)sc.part, p.f_nck, p.f_ck))
  switch (a.dh) {
    case 64: CMB(64); break;
    case 128: CMB(128); break;
    case 256: CMB(256); break;
    default: return hipErrorInvalidValue;
  }
#undef CMB
  return hipGetLastError();
}

hipError_t launch_attn_delta(const bf16* dO, const f16* O, int ld, int B, int T, int H, int dh, float* delta,
                             hipStream_t st) {
  const size_t nd = (size_t)B * T * H;
  MEBP_TIMED(st, "attn_delta", 0.0, (double)nd * (4.0 * dh + 4),
             hipLaunchKernelGGL(k_attn_delta, dim3((unsigned)((nd * (dh / 8) + 255) / 256)), dim3(256), 0, st, dO, O, ld,
                                B, T, H, dh, delta));
  return hipGetLastError();
}

hipError_t launch_attn_bwd(const AttnArgs& a0, float* delta_ws, const SplitScratch& sc, hipStream_t st,
                           hipStream_t aux, hipEvent_t ev_go, hipEvent_t ev_done, bool delta_ready) {
  hipError_t e;
  if (!delta_ready &&
      (e = launch_attn_delta(a0.dO, (const f16*)a0.o, a0.ldq, a0.B, a0.T, a0.Hq, a0.dh, delta_ws, st)) != hipSuccess)
    return e;
  AttnArgs a = a0;
  a.delta = delta_ws;
  // (the kernels address a sequence's rows with 32-bit buffer offsets)
  if ((double)a.T * (a.ldq > a.ldk ? a.ldq : a.ldk) * 2 >= 2147483648.0) return hipErrorInvalidValue;
  const AttnPlan p = attn_plan(a.B, a.T, a.Hq, a.Hkv, a.dh, a.window);
  if ((p.kv_floats + p.q_floats) && (!sc.part || sc.part_floats < p.kv_floats + p.q_floats))
    return hipErrorInvalidValue;
  float* kv_part = sc.part;
  float* q_part = sc.part + p.kv_floats;
  const int nt64 = (a.T + 63) / 64;
  const dim3 gkv(nt64 * (p.kv_nck ? p.kv_nck : 1), a.Hq, a.B), gq(nt64 * (p.q_nck ? p.q_nck : 1), a.Hq, a.B);
  const double pairs = visible_pairs(a.T, a.window) * a.Hq * a.B;
  // algorithmic: dV, dK and dP products in the key-block kernel, dQ in the query-block kernel
  const double f_kv = 6.0 * a.dh * pairs, f_q = 2.0 * a.dh * pairs;
  const double io = (double)a.B * a.T * (a.Hq * a.dh * 2.0 * 2 + a.Hkv * a.dh * 2.0 * 4);
  // dQ depends only on delta and the forward tensors: with an auxiliary stream it runs
  // there while dK / dV run here
  const bool split = aux && ev_go && ev_done;
  hipStream_t sq = split ? aux : st;
  if (split) {
    if ((e = hipEventRecord(ev_go, st)) != hipSuccess) return e;
    if ((e = hipStreamWaitEvent(aux, ev_go, 0)) != hipSuccess) return e;
  }
#define DQ(D, KB, PF) \
  MEBP_TIMED(sq, "attn_bwd_dq", f_q, io, hipLaunchKernelGGL((k_attn_bwd_dq<D, KB, PF>), gq, dim3(256), 0, sq, a, q_part, p.q_nck, p.q_ck))
  switch (a.dh) {
    case 64: DQ(64, 64, true); break;
    case 128: DQ(128, 64, true); break;
    case 256: DQ(256, 32, false); break;
    default: return hipErrorInvalidValue;
  }
#undef DQ
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (p.q_nck) {
    const size_t nr = (size_t)a.B * a.T * a.Hq * (a.dh / 8);
    MEBP_TIMED(sq, "attn_dq_reduce", 0.0, (double)p.q_floats * 4 + (double)a.B * a.T * a.Hq * a.dh * 2,
               hipLaunchKernelGGL(k_attn_dq_reduce, dim3((unsigned)((nr + 255) / 256)), dim3(256), 0, sq, a,
                                  (const float*)q_part, p.q_nck, p.q_ck, a.dh == 256 ? 32 : 64));
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  // head dim 128: 32-key waves (four per workgroup). Head dim 64 keeps the 16-key kernel,
  // which is faster at the short sequences that use it, and 256 too: there dK^T and dV^T
  // alone fill the accumulation registers.
  if (a.dh == 128) {
    const dim3 gkv32((a.T + 127) / 128, a.Hq, a.B);
    MEBP_TIMED(st, "attn_bwd_dkdv", f_kv, io,
               hipLaunchKernelGGL((k_attn_bwd_kv32<128, 4>), gkv32, dim3(256), 0, st, a, kv_part));
  } else switch (a.dh) {
    case 64:
      MEBP_TIMED(st, "attn_bwd_dkdv", f_kv, io,
                 hipLaunchKernelGGL((k_attn_bwd_dkdv<64, 64>), gkv, dim3(256), 0, st, a, kv_part, p.kv_nck, p.kv_cq));
      break;
    case 256:
      if (!p.kv_nck) {
        // 64 keys per workgroup: two wave pairs of 32 keys, one wave per SIMD
        const dim3 gp((a.T + 63) / 64, a.Hq, a.B);
        MEBP_TIMED(st, "attn_bwd_dkdv", f_kv, io,
                   hipLaunchKernelGGL((k_attn_bwd_kv32p<2>), gp, dim3(256), 0, st, a, kv_part));
      } else {
        MEBP_TIMED(st, "attn_bwd_dkdv", f_kv, io,
                   hipLaunchKernelGGL((k_attn_bwd_dkdv<256, 32>), gkv, dim3(256), 0, st, a, kv_part, p.kv_nck, p.kv_cq));
      }
      break;
    default: return hipErrorInvalidValue;
  }
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (split) {
    if ((e = hipEventRecord(ev_done, aux)) != hipSuccess) return e;
  }
  if (p.kv_floats) {
    const size_t nr = (size_t)a.B * a.T * a.Hkv * (a.dh / 8);
    MEBP_TIMED(st, "attn_dkdv_reduce", 0.0, (double)p.kv_floats * 4 + (double)a.B * a.T * a.Hkv * a.dh * 4,
               hipLaunchKernelGGL(k_attn_dkdv_reduce, dim3((unsigned)((nr + 255) / 256)), dim3(256), 0, st, a,
                                  (const float*)kv_part, p.kv_nck, p.kv_cq));
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return split ? hipStreamWaitEvent(st, ev_done, 0) : hipSuccess;
}

}  // namespace mebp
