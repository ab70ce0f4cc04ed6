// Large-tile int4 group-dequant GEMMs for many tokens (M = B*T in the thousands): the same
// products as gemm_q4.hip (forward "NT" and transposed "TN", Algorithm 1's lazily
// decompressed weights fused into the operand load), with a tiling sized for MFMA
// throughput rather than for latency.
//
// One 256 x BN output tile per 256-thread workgroup (BN = 256 or 128), 2 x 2 waves of
// 128 x BN/2, v_mfma_f32_32x32x16 (fp16 operands forward, bf16 backward), K step 64.
// Per wave and K step the fragments read from LDS are (128 + BN/2) x 64 16-bit values for
// 128 x BN/2 x 64 MACs: 32 MACs per LDS byte at BN = 256 (16 for the 128 x 128 tiles of
// gemm_q4.hip), so LDS reads take about half of the MFMA time at the chip's 128 B/clk/CU.
// One workgroup per CU (up to 144 KB of LDS, 256 fp32 accumulators per lane). Pipeline:
// the global loads of K tile t+2 are issued before the MFMAs of tile t, and tile t+1 is
// decompressed from registers into the other LDS buffer after them.
//
// MFMA 32x32x16 lane layout: lane l supplies A[l%32][8(l/32) .. +8] and
// B[8(l/32) .. +8][l%32]; accumulator element q of lane l is D[8(q/4) + 4(l/32) + q%4][l%32].
//
// The LoRA up-projection (unsplit case) is three extra bf16 MFMAs per accumulator tile on
// the fp32 factors split into bf16 hi + lo parts (hi*hi + hi*lo + lo*hi, relative error
// below 2^-16), so no scalar epilogue loop is needed.
#include "device_common.h"
#include "mebp_internal.h"

namespace mebp {
namespace {

constexpr int BM = 256, BK = 64, LDT = BK + 8, NTH = 256;
typedef uint16_t u16;
typedef float f32x16 __attribute__((ext_vector_type(16)));

template <int N>
struct IC {
  static constexpr int value = N;
};

template <class Op>
DEV f32x16 mfma32(uint4 a, uint4 b, f32x16 c) {
  if constexpr (__is_same(Op, OpF16))
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), c, 0, 0,
                                                  0);
  else
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c, 0,
                                                   0, 0);
}

template <int NJ>
DEV void zero_acc(f32x16 (&acc)[4][NJ]) {
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < NJ; ++j)
#pragma unroll
      for (int q = 0; q < 16; ++q) acc[i][j][q] = 0.f;
}

// tile-local row of accumulator element q of row block i, and column of column block j
DEV int acc_row(int wm, int i, int q, int lane) { return wm * 128 + 32 * i + 8 * (q >> 2) + 4 * (lane >> 5) + (q & 3); }
template <int NJ>
DEV int acc_col(int wn, int j, int lane) {
  return wn * 32 * NJ + 32 * j + (lane & 31);
}

// One K tile of the wave's 128 x 32NJ block from the LDS tiles (row pitch LDT; A rows are
// M, B rows are N, both K-contiguous).
template <class Op, int NJ>
DEV void mma_tile(const u16* As, const u16* Bs, int wm, int wn, int lane, f32x16 (&acc)[4][NJ]) {
  const int r = lane & 31, kh = 8 * (lane >> 5);
  const u16* pa = As + (wm * 128 + r) * LDT + kh;
  const u16* pb = Bs + (wn * 32 * NJ + r) * LDT + kh;
#pragma unroll
  for (int ks = 0; ks < BK; ks += 16) {
    uint4 af[4], bfr[NJ];
#pragma unroll
    for (int i = 0; i < 4; ++i) af[i] = *(const uint4*)(pa + 32 * i * LDT + ks);
#pragma unroll
    for (int j = 0; j < NJ; ++j) bfr[j] = *(const uint4*)(pb + 32 * j * LDT + ks);
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < NJ; ++j) acc[i][j] = mfma32<Op>(af[i], bfr[j], acc[i][j]);
  }
}

// v (8 fp32) -> bf16 hi and lo parts with v ~ hi + lo
DEV void split_bf16(const float (&v)[8], uint4& hi, uint4& lo) {
  float h[8], l[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    h[e] = (float)(bf16)v[e];
    l[e] = v[e] - h[e];
  }
  hi = make_uint4(pack_bf16x2(h[0], h[1]), pack_bf16x2(h[2], h[3]), pack_bf16x2(h[4], h[5]), pack_bf16x2(h[6], h[7]));
  lo = make_uint4(pack_bf16x2(l[0], l[1]), pack_bf16x2(l[2], l[3]), pack_bf16x2(l[4], l[5]), pack_bf16x2(l[6], l[7]));
}

// acc += s * U[m][:r] . V(col)[:r] for the wave's block: U fp32 [M][r] (rows from mrow0),
// V(col)[q] = V[col * vcol + q * vq] fp32 (columns from ccol0, < ncols); r = 8 or 16 (the
// rank is the MFMA's K = 16; lanes past r supply zeros). All loads go through buffer
// resources (rows past M, columns past ncols read 0) and are issued before any use, so
// they overlap instead of waiting one by one.
template <int NJ>
DEV void lora_mfma(f32x16 (&acc)[4][NJ], const float* U, int r, int mrow0, int M, float s, const float* V,
                   int vcol, int vq, int ccol0, int ncols, int lane) {
  const int q0 = 8 * (lane >> 5);
  const bool keep = q0 < r;  // select, not multiply: a neighbouring row's value may be non-finite
  const rsrc_t rU = make_rsrc(U, (size_t)M * r * 4);
  const rsrc_t rV = make_rsrc(V, (size_t)((ncols - 1) * vcol + (r - 1) * vq + 1) * 4);
  float vv[NJ][8], uu[4][8];
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    const int c = ccol0 + 32 * j + (lane & 31);
    const bool cok = c < ncols;
#pragma unroll
    for (int e = 0; e < 8; ++e)
      vv[j][e] = __builtin_bit_cast(float, bload32(rV, cok ? (uint32_t)((c * vcol + (q0 + e) * vq) * 4) : 0xffffffffu));
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = mrow0 + 32 * i + (lane & 31);
    const uint4 a0 = bload128(rU, (uint32_t)((m * r + q0) * 4)), a1 = bload128(rU, (uint32_t)((m * r + q0 + 4) * 4));
    uu[i][0] = __builtin_bit_cast(float, a0.x); uu[i][1] = __builtin_bit_cast(float, a0.y);
    uu[i][2] = __builtin_bit_cast(float, a0.z); uu[i][3] = __builtin_bit_cast(float, a0.w);
    uu[i][4] = __builtin_bit_cast(float, a1.x); uu[i][5] = __builtin_bit_cast(float, a1.y);
    uu[i][6] = __builtin_bit_cast(float, a1.z); uu[i][7] = __builtin_bit_cast(float, a1.w);
  }
  uint4 bh[NJ], bl[NJ];
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    float v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = keep ? vv[j][e] : 0.f;
    split_bf16(v, bh[j], bl[j]);
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    float u[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) u[e] = keep ? s * uu[i][e] : 0.f;
    uint4 ah, al;
    split_bf16(u, ah, al);
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      acc[i][j] = mfma32<OpBF16>(ah, bh[j], acc[i][j]);
      acc[i][j] = mfma32<OpBF16>(ah, bl[j], acc[i][j]);
      acc[i][j] = mfma32<OpBF16>(al, bh[j], acc[i][j]);
    }
  }
}

// split-K: the workgroup's partial tile into the plane of its split ([M][ldp] fp32, columns
// from c0), reduced in split order by a finalize kernel
template <int NJ>
DEV void store_partial(const f32x16 (&acc)[4][NJ], float* plane, int M, int ldp, int ncols, int m0, int c0, int wm,
                       int wn, int lane) {
  auto put = [&](auto FULL_) {
    constexpr bool FULL = decltype(FULL_)::value;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        const int m = m0 + acc_row(wm, i, q, lane);
        if (!FULL && m >= M) continue;
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
          const int c = acc_col<NJ>(wn, j, lane);
          if (!FULL && c >= ncols) continue;
          plane[(size_t)m * ldp + c0 + c] = acc[i][j][q];
        }
      }
  };
  if (m0 + BM <= M && 64 * NJ <= ncols)
    put(IC<1>{});
  else
    put(IC<0>{});
}

// A-operand staging: 8 chunks of 8 16-bit elements per thread; chunk c = tid + 256 i covers
// row c >> 3 (= tid/8 + 32 i), columns (c & 7) * 8 .. +8 of the 256 x 64 tile.
DEV void store_a_tile(u16* As, int tid, const uint4 (&ra)[8]) {
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int c = tid + NTH * i;
    *(uint4*)(As + (c >> 3) * LDT + (c & 7) * 8) = ra[i];
  }
}

// ------------------------------------------------------------------------------ forward
// C[m][n] = sum_k X[m][k] W[n][k] (+ s u B^T + resid), fp16 operands.
//
// The weight operand does not go through LDS: for MFMA column j of its block a lane needs
// 8 reduction indices of one weight row, i.e. one dword of codes. Within a K tile of 64 a
// lane of half h (= lane / 32) takes the four consecutive dwords 4h .. 4h+3 of its row (one
// 16-byte load, one 32-group, one scale) and uses dword 4h+s in substep s; the activation
// fragments read from LDS follow the same assignment of reduction indices. Decompression is
// done with packed fp16 arithmetic, which orders the eight values of a dword as
// (k0,k4),(k1,k5),(k2,k6),(k3,k7); activation chunks are stored into LDS in that order too.
// Each wave thus decompresses only the weights it multiplies, and LDS carries the
// activation tile alone.

// 8 int4 codes (two's complement, element i in bits 4i..4i+3) times scale into fp16 pairs
// (k0,k4),(k1,k5),(k2,k6),(k3,k7): 0x6400 | (q + 8) is the fp16 value 1024 + q + 8, so one
// packed subtraction of 1032 gives q exactly and one packed multiply rounds q * s to nearest.
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
DEV uint4 dequant8_paired(uint32_t w, f16x2 s2) {
  const uint32_t x = w ^ 0x88888888u;
  const f16x2 off = {(_Float16)1032.0f, (_Float16)1032.0f};
  uint32_t o[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const uint32_t t = ((x >> (4 * j)) & 0x000F000Fu) | 0x64006400u;
    const f16x2 v = (__builtin_bit_cast(f16x2, t) - off) * s2;
    o[j] = __builtin_bit_cast(uint32_t, v);
  }
  return make_uint4(o[0], o[1], o[2], o[3]);
}

// (k0..k7) -> (k0,k4),(k1,k5),(k2,k6),(k3,k7), the order of dequant8_paired
DEV uint4 pair_order(uint4 d) {
  return make_uint4(perm_lo16(d.x, d.z), perm_hi16(d.x, d.z), perm_lo16(d.y, d.w), perm_hi16(d.y, d.w));
}

// The segment's fields as scalar values: indexing the argument struct with a run-time
// segment number would make the compiler copy it to scratch memory.
DEV NtSeg pick_seg(const NtArgs& a, int s) {
  NtSeg r;
#define PICK(f) r.f = s == 0 ? a.seg[0].f : (s == 1 ? a.seg[1].f : a.seg[2].f)
  PICK(q4);
  PICK(scale);
  PICK(N);
  PICK(tile0);
  PICK(col0);
  PICK(lora_u);
  PICK(lora_B);
  PICK(out);
  PICK(ldo);
  PICK(resid);
  PICK(ldr);
#undef PICK
  r.rope = 0;
  r.item0 = 0;
  return r;
}

// Epilogue of the forward large-tile kernels: logits statistics, split-K partial planes, or
// LoRA up-projection + residual + fp16 / fp32 store of the wave's 128 x 32NJ block.
template <int BN, int WNW, int EPI>
DEV void nt_big_epilogue(f32x16 (&acc)[4][BN / (32 * WNW)], const NtArgs& a, const NtSeg& sg, int m0, int n0,
                         int wcol0, int wm, int wn, int lane, int z, int S) {
  constexpr int NJ = BN / (32 * WNW);
  const int Nn = sg.N;
  if constexpr (EPI == NT_LOGITS) {
    // every wave covers one statistics tile of 32 NJ = 64 columns: per row its max, its
    // sum of exp(v - max), the logits minus that max (fp16), and the fp32 target logit
    static_assert(32 * NJ == 64, "statistics tiles are 64 columns wide");
    _Float16* out = (_Float16*)sg.out;
    const int cw0 = wcol0;
    const int stile = cw0 / (32 * NJ);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        const int m = m0 + acc_row(wm, i, q, lane);
        float mx = -INFINITY;
#pragma unroll
        for (int j = 0; j < NJ; ++j)
          if (cw0 + 32 * j + (lane & 31) < Nn) mx = fmaxf(mx, acc[i][j][q]);
#pragma unroll
        for (int o = 1; o < 32; o <<= 1) mx = fmaxf(mx, __shfl_xor(mx, o, 64));
        const int tg = m < a.M ? a.tgt[m] : -1;
        float se = 0.f;
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
          const int n = cw0 + 32 * j + (lane & 31);
          if (n < Nn) {
            const float v = acc[i][j][q];
            se += __expf(v - mx);
            if (m < a.M) {
              out[(size_t)m * sg.ldo + n] = (_Float16)(v - mx);
              if (n + a.vbase == tg) a.tgt_logit[m] = v;
            }
          }
        }
#pragma unroll
        for (int o = 1; o < 32; o <<= 1) se += __shfl_xor(se, o, 64);
        if ((lane & 31) == 0 && m < a.M && cw0 < Nn) a.stats[(size_t)m * a.ntiles + stile] = make_float2(mx, se);
      }
    }
    return;
  } else {
    if (S > 1) {
      store_partial<NJ>(acc, a.part + (size_t)z * a.M * a.ldp, a.M, a.ldp, Nn - n0, m0, sg.col0 + n0, wm, wn, lane);
      return;
    }
    if (sg.lora_B)
      lora_mfma<NJ>(acc, sg.lora_u, a.r, m0 + wm * 128, a.M, a.lora_s, sg.lora_B, a.r, 1, wcol0, Nn, lane);
    auto put = [&](auto FULL_, auto RES_) {
      constexpr bool FULL = decltype(FULL_)::value, RES = decltype(RES_)::value;
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int q = 0; q < 16; ++q) {
          const int m = m0 + acc_row(wm, i, q, lane);
          if (!FULL && m >= a.M) continue;
#pragma unroll
          for (int j = 0; j < NJ; ++j) {
            const int n = n0 + acc_col<NJ>(wn, j, lane);
            if (!FULL && n >= Nn) continue;
            float v = acc[i][j][q];
            if constexpr (RES) v += sg.resid[(size_t)m * sg.ldr + n];
            if constexpr (EPI == NT_STORE_F16)
              ((f16*)sg.out)[(size_t)m * sg.ldo + n] = (f16)v;
            else
              ((float*)sg.out)[(size_t)m * sg.ldo + n] = v;
          }
        }
    };
    const bool full = m0 + BM <= a.M && n0 + BN <= Nn;
    if (sg.resid) {
      if (full) put(IC<1>{}, IC<1>{}); else put(IC<0>{}, IC<1>{});
    } else {
      if (full) put(IC<1>{}, IC<0>{}); else put(IC<0>{}, IC<0>{});
    }
  }
}

// fp16 / fp32 store (LoRA up-projection and residual included) of a wave's 128 x 64 block
// of the large-tile forward kernels through LDS: per 32-row block the accumulators (MFMA layout) go into the
// wave's own 32 x 68 fp32 region, and each lane reads back 8 consecutive columns of a row
// and stores them with 16-byte accesses (a wave instruction covers 8 whole row segments)
// instead of 2- or 4-byte stores in the MFMA layout. The residual rows of a block are all
// loaded before its accumulators are staged. Requires N % 8 == 0 and 16-byte aligned rows.
// LM-head logits epilogue through a per-wave LDS region (32 x 68 fp32): for each 32-row block
// of the wave's 128 x 64 tile, lane (row r = 8p + lane / 8, columns 8 (lane % 8) ..) takes 8
// consecutive values of one row, so that the statistics of a row's 64-column tile reduce over
// the 8 lanes that hold it (three shuffle steps) and its fp16 values leave as one 16-byte store.
// Per row and tile: max, sum of exp(v - max), the values minus the max (fp16), and the fp32
// logit of the target (vocabulary columns are offset by vbase). The segment width is a
// multiple of 32, so an 8-column group is either wholly inside it or wholly past it.
DEV void nt_lds_logits_store(f32x16 (&acc)[4][2], const NtArgs& a, const NtSeg& sg, int mw0, int wcol0, int lane,
                             float* ep) {
  constexpr int LDE = 68;
  const int rr = lane >> 3, ch = lane & 7, n = wcol0 + 8 * ch, Nn = sg.N;
  const bool nok = n < Nn, tile_ok = wcol0 < Nn;
  const int stile = wcol0 / 64;
  _Float16* out = (_Float16*)sg.out;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
#pragma unroll
    for (int q = 0; q < 16; ++q)
#pragma unroll
      for (int j = 0; j < 2; ++j) ep[(8 * (q >> 2) + 4 * (lane >> 5) + (q & 3)) * LDE + 32 * j + (lane & 31)] = acc[i][j][q];
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      const int r = 8 * p + rr, m = mw0 + 32 * i + r;
      const float4 v0 = *(const float4*)(ep + r * LDE + 8 * ch), v1 = *(const float4*)(ep + r * LDE + 8 * ch + 4);
      const float v[8] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w};
      float mx = -INFINITY;
      if (nok) {
#pragma unroll
        for (int e = 0; e < 8; ++e) mx = fmaxf(mx, v[e]);
      }
      mx = fmaxf(mx, __shfl_xor(mx, 1, 64));
      mx = fmaxf(mx, __shfl_xor(mx, 2, 64));
      mx = fmaxf(mx, __shfl_xor(mx, 4, 64));
      float se = 0.f;
      if (nok) {
#pragma unroll
        for (int e = 0; e < 8; ++e) se += __expf(v[e] - mx);
      }
      se += __shfl_xor(se, 1, 64);
      se += __shfl_xor(se, 2, 64);
      se += __shfl_xor(se, 4, 64);
      if (m < a.M) {
        if (nok) {
          const uint4 o = make_uint4(pack_f16x2(v[0] - mx, v[1] - mx), pack_f16x2(v[2] - mx, v[3] - mx),
                                     pack_f16x2(v[4] - mx, v[5] - mx), pack_f16x2(v[6] - mx, v[7] - mx));
          *(uint4*)(out + (size_t)m * sg.ldo + n) = o;
          const int tg = a.tgt[m] - a.vbase - n;
          if (tg >= 0 && tg < 8) a.tgt_logit[m] = v[tg];
        }
        if (ch == 0 && tile_ok) a.stats[(size_t)m * a.ntiles + stile] = make_float2(mx, se);
      }
    }
  }
}

// lora_mfma with u and B already in LDS (rows of r floats: the tile's u rows from urow0, its
// B rows from bcol0), copied there while the main loop ran
template <int NJ>
DEV void lora_mfma_lds(f32x16 (&acc)[4][NJ], const float* Us, const float* Bs, int r, int urow0, float s, int bcol0,
                       int lane) {
  const int q0 = 8 * (lane >> 5);
  const bool keep = q0 < r;  // select, not multiply (see lora_mfma)
  const int qe = keep ? q0 : 0;
  uint4 bh[NJ], bl[NJ];
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    const float* p = Bs + (bcol0 + 32 * j + (lane & 31)) * r + qe;
    const float4 x0 = *(const float4*)p, x1 = *(const float4*)(p + 4);
    float v[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = keep ? v[e] : 0.f;
    split_bf16(v, bh[j], bl[j]);
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float* p = Us + (urow0 + 32 * i + (lane & 31)) * r + qe;
    const float4 x0 = *(const float4*)p, x1 = *(const float4*)(p + 4);
    float u[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
#pragma unroll
    for (int e = 0; e < 8; ++e) u[e] = keep ? s * u[e] : 0.f;
    uint4 ah, al;
    split_bf16(u, ah, al);
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      acc[i][j] = mfma32<OpBF16>(ah, bh[j], acc[i][j]);
      acc[i][j] = mfma32<OpBF16>(ah, bl[j], acc[i][j]);
      acc[i][j] = mfma32<OpBF16>(al, bh[j], acc[i][j]);
    }
  }
}

// LORA_LDS: the tile's u and B rows are in LDS at lora_lds (u rows from urow0 and B rows
// from bcol0 for this wave), else they are read from global memory
template <int EPI, bool LORA_LDS = false>
DEV void nt_lds_store(f32x16 (&acc)[4][2], const NtArgs& a, const NtSeg& sg, int mw0, int wcol0, int lane,
                      float* ep, const float* lora_lds = nullptr, int urow0 = 0, int bcol0 = 0) {
  constexpr int LDE = 68;
  if (sg.lora_B) {
    if constexpr (LORA_LDS)
      lora_mfma_lds<2>(acc, lora_lds, lora_lds + BM * 16, a.r, urow0, a.lora_s, bcol0, lane);
    else
      lora_mfma<2>(acc, sg.lora_u, a.r, mw0, a.M, a.lora_s, sg.lora_B, a.r, 1, wcol0, sg.N, lane);
  }
  const int rr = lane >> 3, ch = lane & 7, n = wcol0 + 8 * ch;
  const bool nok = n < sg.N;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    float4 res[4][2];
    if (sg.resid) {
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        const int m = mw0 + 32 * i + 8 * p + rr;
        const bool ok = nok && m < a.M;
        const float* src = sg.resid + (ok ? (size_t)m * sg.ldr + n : 0);
        res[p][0] = ok ? *(const float4*)src : make_float4(0.f, 0.f, 0.f, 0.f);
        res[p][1] = ok ? *(const float4*)(src + 4) : make_float4(0.f, 0.f, 0.f, 0.f);
      }
    }
#pragma unroll
    for (int q = 0; q < 16; ++q)
#pragma unroll
      for (int j = 0; j < 2; ++j) ep[(8 * (q >> 2) + 4 * (lane >> 5) + (q & 3)) * LDE + 32 * j + (lane & 31)] = acc[i][j][q];
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      const int r = 8 * p + rr, m = mw0 + 32 * i + r;
      float4 v0 = *(const float4*)(ep + r * LDE + 8 * ch), v1 = *(const float4*)(ep + r * LDE + 8 * ch + 4);
      if (sg.resid) {
        v0.x += res[p][0].x; v0.y += res[p][0].y; v0.z += res[p][0].z; v0.w += res[p][0].w;
        v1.x += res[p][1].x; v1.y += res[p][1].y; v1.z += res[p][1].z; v1.w += res[p][1].w;
      }
      if (nok && m < a.M) {
        if constexpr (EPI == NT_STORE_F16) {
          const uint4 o = make_uint4(pack_f16x2(v0.x, v0.y), pack_f16x2(v0.z, v0.w), pack_f16x2(v1.x, v1.y),
                                     pack_f16x2(v1.z, v1.w));
          *(uint4*)((f16*)sg.out + (size_t)m * sg.ldo + n) = o;
        } else {
          float* dst = (float*)sg.out + (size_t)m * sg.ldo + n;
          *(float4*)dst = v0;
          *(float4*)(dst + 4) = v1;
        }
      }
    }
  }
}

// Gated MLP epilogue (the model's MLP: z = act(g) * u): the tile holds 128 gate
// and the same 128 up features, waves 0, 1 the gate columns and waves 2, 3 the up columns
// (wave w and w ^ 2 cover the same 64 features). Each wave stages a 32-row chunk of its
// fp32 outputs in its own LDS region (ep); after a barrier the gate wave forms z for the
// chunk's first 16 rows and the up wave for the last 16, reading g and u from both regions,
// with the same fp16 roundings as the stand-alone activation kernel (g and u rounded to
// fp16, z = fp16(act(g) * u)). Used where z alone is needed (the forward pass); g and u are
// not stored. KIND is the activation (0 SiLU, 1 tanh-GELU).
template <int KIND>
DEV void nt_lds_store_gated(f32x16 (&acc)[4][2], const NtArgs& a, const NtSeg& sg, int mw0, int f0w, int lane,
                            float* ep, const float* pep, const float* Us, const float* Bs, int urow0, int bcol0,
                            int is_up) {
  constexpr int LDE = 68;
  if (sg.lora_B) lora_mfma_lds<2>(acc, Us, Bs, a.r, urow0, a.lora_s, bcol0, lane);
  const int rr = lane >> 3, ch = lane & 7, n = f0w + 8 * ch;
  const bool nok = n < sg.N;
  const float* gsrc = is_up ? pep : ep;
  const float* usrc = is_up ? ep : pep;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
#pragma unroll
    for (int q = 0; q < 16; ++q)
#pragma unroll
      for (int j = 0; j < 2; ++j) ep[(8 * (q >> 2) + 4 * (lane >> 5) + (q & 3)) * LDE + 32 * j + (lane & 31)] = acc[i][j][q];
    __syncthreads();  // the partner wave's chunk is staged
#pragma unroll
    for (int p = 0; p < 2; ++p) {
      const int r = 16 * is_up + 8 * p + rr, m = mw0 + 32 * i + r;
      const float4 g0 = *(const float4*)(gsrc + r * LDE + 8 * ch), g1 = *(const float4*)(gsrc + r * LDE + 8 * ch + 4);
      const float4 u0 = *(const float4*)(usrc + r * LDE + 8 * ch), u1 = *(const float4*)(usrc + r * LDE + 8 * ch + 4);
      const uint32_t gq[4] = {pack_f16x2(g0.x, g0.y), pack_f16x2(g0.z, g0.w), pack_f16x2(g1.x, g1.y), pack_f16x2(g1.z, g1.w)};
      const uint32_t uq[4] = {pack_f16x2(u0.x, u0.y), pack_f16x2(u0.z, u0.w), pack_f16x2(u1.x, u1.y), pack_f16x2(u1.z, u1.w)};
      uint32_t o[4];
#pragma unroll
      for (int t = 0; t < 4; ++t)
        o[t] = pack_f16x2(act_k<KIND>(f16_lo(gq[t])) * f16_lo(uq[t]), act_k<KIND>(f16_hi(gq[t])) * f16_hi(uq[t]));
      if (nok && m < a.M) *(uint4*)(a.z_out + (size_t)m * sg.N + n) = make_uint4(o[0], o[1], o[2], o[3]);
    }
    __syncthreads();  // both waves are done with the chunk before the next one is staged
  }
}

// WNW waves along n (2 or 4), two along m: 128 x WNW threads, each wave 128 x BN/WNW. With
// four (512 threads) two waves share each SIMD, so one wave's decompression (VALU) runs
// beside the other's MFMAs.
// VEC: fp16 / fp32 outputs through nt_lds_store (one split, N % 8 == 0, 16-byte aligned rows).
template <int BN, int WNW, int EPI, bool VEC>
__global__ __launch_bounds__(128 * WNW, 1) void k_gemm_nt_big(const NtArgs a) {
  constexpr int NT = 128 * WNW;
  constexpr int NJ = BN / (32 * WNW);  // 32-column blocks per wave
  constexpr int NA = 2048 / NT;        // 16-byte activation chunks per thread and K tile
  __shared__ __attribute__((aligned(16))) u16 As2[2][BM * LDT];
  // the wave index is wave-uniform; saying so keeps the weight resources in SGPRs
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WNW, wn = wave % WNW, h = lane >> 5;
  const int nt = blockIdx.x;
  int s = 0;
  if (a.nseg > 1 && nt >= a.seg[1].tile0) s = 1;
  if (a.nseg > 2 && nt >= a.seg[2].tile0) s = 2;
  const NtSeg sg = pick_seg(a, s);
  const int n0 = (nt - sg.tile0) * BN, m0 = blockIdx.y * BM;
  const int K = a.K, Nn = sg.N, Kh = K >> 1;
  const int nk = (K + BK - 1) / BK, kgroups = (K + 31) >> 5;
  const int z = blockIdx.z, S = gridDim.z;
  const int kt_begin = (int)((long long)nk * z / S), kt_end = (int)((long long)nk * (z + 1) / S);

  const rsrc_t rA = make_rsrc((const u16*)a.X + (size_t)m0 * a.lda, (size_t)min(BM, a.M - m0) * a.lda * 2);
  const int wcol0 = n0 + wn * 32 * NJ;  // first weight row (output column) of this wave
  const int wrows = max(0, min(32 * NJ, Nn - wcol0));
  const rsrc_t rB = make_rsrc(sg.q4 + (size_t)min(wcol0, Nn) * Kh, (size_t)wrows * Kh);
  const rsrc_t rS = make_rsrc(sg.scale + (size_t)min(wcol0, Nn) * kgroups, (size_t)wrows * kgroups * 2);
  uint32_t offA[NA];
#pragma unroll
  for (int i = 0; i < NA; ++i) {
    const int c = tid + NT * i;
    offA[i] = (uint32_t)(((c >> 3) * a.lda + (c & 7) * 8) * 2);
  }
  const uint32_t offB = (uint32_t)((lane & 31) * Kh + 16 * h), offS = (uint32_t)(((lane & 31) * kgroups + h) * 2);

  uint4 ra[2][NA];
  uint4 rb[2][NJ];
  uint32_t rsc[2][NJ];  // raw fp16 scale bits
  f32x16 acc[4][NJ];
  zero_acc(acc);

  auto run = [&](auto TAIL_) {
    constexpr bool TAIL = decltype(TAIL_)::value;
    auto gload_a = [&](auto S_, int kt) {
      constexpr int st = decltype(S_)::value;
      const int k0 = kt * BK;
#pragma unroll
      for (int i = 0; i < NA; ++i) ra[st][i] = bload128(rA, offA[i] + 2 * k0);
      if constexpr (TAIL) {
        if (k0 + BK > K) {  // zero what lies past the reduction length
#pragma unroll
          for (int i = 0; i < NA; ++i)
            if (((tid + NT * i) & 7) * 8 + k0 >= K) ra[st][i] = make_uint4(0, 0, 0, 0);
        }
      }
    };
    auto gload_b = [&](auto S_, int kt) {
      constexpr int st = decltype(S_)::value;
      const int k0 = kt * BK;
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        rb[st][j] = bload128(rB, offB + (uint32_t)(32 * j * Kh) + (k0 >> 1));
        rsc[st][j] = bload16(rS, offS + (uint32_t)(32 * j * kgroups * 2) + 2 * (k0 >> 5));
      }
      if constexpr (TAIL) {
        if (k0 + BK > K) {
          const int kb = k0 + 32 * h;
#pragma unroll
          for (int j = 0; j < NJ; ++j) {
            if (kb >= K) rsc[st][j] = 0u;
            if (kb + 0 >= K) rb[st][j].x = 0u;
            if (kb + 8 >= K) rb[st][j].y = 0u;
            if (kb + 16 >= K) rb[st][j].z = 0u;
            if (kb + 24 >= K) rb[st][j].w = 0u;
          }
        }
      }
    };
    auto sstore = [&](auto S_, auto B_) {
      constexpr int st = decltype(S_)::value, bf = decltype(B_)::value;
#pragma unroll
      for (int i = 0; i < NA; ++i) {
        const int c = tid + NT * i;
        *(uint4*)(As2[bf] + (c >> 3) * LDT + (c & 7) * 8) = pair_order(ra[st][i]);
      }
    };
    // the MFMAs of one K tile: substep t uses chunk 4h + t of the lane's reduction range
    auto mma = [&](auto S_, auto B_) {
      constexpr int st = decltype(S_)::value, bf = decltype(B_)::value;
      const u16* pa = As2[bf] + (wm * 128 + (lane & 31)) * LDT + 32 * h;
      f16x2 sc[NJ];
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        const _Float16 v = __builtin_bit_cast(_Float16, (uint16_t)rsc[st][j]);
        sc[j] = f16x2{v, v};
      }
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        uint4 af[4], bfr[NJ];
#pragma unroll
        for (int i = 0; i < 4; ++i) af[i] = *(const uint4*)(pa + 32 * i * LDT + 8 * t);
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
          const uint32_t w = t == 0 ? rb[st][j].x : t == 1 ? rb[st][j].y : t == 2 ? rb[st][j].z : rb[st][j].w;
          bfr[j] = dequant8_paired(w, sc[j]);
        }
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < NJ; ++j) acc[i][j] = mfma32<OpF16>(af[i], bfr[j], acc[i][j]);
      }
    };
    // step for tile k (I = parity): loads of tile k+2 into the A stage tile k vacated, the
    // MFMAs of tile k (LDS buffer I, weights of stage I), tile k+1's activations into the
    // other LDS buffer, one barrier. The weight stage of tile k is consumed by the MFMAs, so
    // tile k+2's weights are loaded after them.
    auto step = [&](auto I_, int k) {
      constexpr int I = decltype(I_)::value;
      const int kn = min(k + 2, kt_end - 1);
      gload_a(IC<I>{}, kn);
      mma(IC<I>{}, IC<I>{});
      gload_b(IC<I>{}, kn);
      sstore(IC<1 - I>{}, IC<1 - I>{});
      __syncthreads();
    };
    gload_a(IC<0>{}, kt_begin);
    gload_b(IC<0>{}, kt_begin);
    gload_a(IC<1>{}, min(kt_begin + 1, kt_end - 1));
    gload_b(IC<1>{}, min(kt_begin + 1, kt_end - 1));
    sstore(IC<0>{}, IC<0>{});
    __syncthreads();
    int k = kt_begin;
    for (; k + 2 <= kt_end; k += 2) {
      step(IC<0>{}, k);
      step(IC<1>{}, k + 1);
    }
    if (k < kt_end) step(IC<0>{}, k);
  };
  if (kt_begin < kt_end) {
    if (K % BK)
      run(IC<1>{});
    else
      run(IC<0>{});
  }

  if constexpr (VEC && EPI != NT_LOGITS && NJ == 2) {
    __syncthreads();  // every wave is done with the main loop's LDS tiles
    nt_lds_store<EPI>(acc, a, sg, m0 + wm * 128, wcol0, lane, reinterpret_cast<float*>(&As2[0][0]) + wave * 32 * 68);
  } else {
    nt_big_epilogue<BN, WNW, EPI>(acc, a, sg, m0, n0, wcol0, wm, wn, lane, z, S);
  }
}


// ---------------------------------------------------------------- forward, LDS-direct tiles
// Natural-order decompression: 8 int4 codes k0..k7 of a dword times scale into fp16 pairs
// (k0,k1),(k2,k3),(k4,k5),(k6,k7). Offset-binary nibbles (code ^ 8) of the even and the odd
// elements are gathered into bytes, a byte permute places one even and one odd code in the
// two halves, 0x6400 | (q + 8) is the fp16 value 1024 + q + 8, and one packed subtraction of
// 1032 and one packed multiply give q exactly and then q * s rounded to nearest.
DEV uint4 dequant8_natural(uint32_t w, f16x2 s2) {
  const uint32_t ev = (w & 0x0F0F0F0Fu) ^ 0x08080808u;         // k0, k2, k4, k6
  const uint32_t od = ((w >> 4) & 0x0F0F0F0Fu) ^ 0x08080808u;  // k1, k3, k5, k7
  const f16x2 off = {(_Float16)1032.0f, (_Float16)1032.0f};
  uint32_t o[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    // byte 0 <- even byte j, byte 2 <- odd byte j, bytes 1 and 3 <- 0
    const uint32_t t = __builtin_amdgcn_perm(od, ev, (uint32_t)j | 0x0C00u | ((4u + j) << 16) | 0x0C000000u) | 0x64006400u;
    o[j] = __builtin_bit_cast(uint32_t, (__builtin_bit_cast(f16x2, t) - off) * s2);
  }
  return make_uint4(o[0], o[1], o[2], o[3]);
}

// vmcnt-only wait (expcnt and lgkmcnt left open), gfx9 encoding
template <int N>
DEV void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// Forward product with 256 x 256 tiles, K step 64, on NW waves: 4 waves of 256 x 64 (one
// wave per SIMD, 256 accumulator registers each; the fp16 and fp32 outputs) or 8 waves of
// 128 x 64 (2 along m x 4 along n; the LM head's logits, whose epilogue takes 128-row waves).
// With 4 waves each weight column block is decompressed by one wave instead of two, which
// halves the decompression's VALU work per MFMA: 5-6 % faster than 8 waves on the Gemma3-4B
// shapes. The activation tile goes from global memory straight into LDS (buffer loads
// with the LDS flag: no staging registers, no LDS stores) through a ring of three stages
// filled two K tiles ahead. A stage holds the 256 x 64 fp16 tile as 128-byte rows whose
// eight 16-byte chunks are stored at position chunk ^ ((row / 2) % 8), so that the MFMA
// fragment reads (32 rows, one chunk each) spread over all banks. The weights are loaded into
// registers, also two tiles ahead, and decompressed by each wave for its own columns.
//
// W16: the weights are plain 16-bit values [N][K] (seg.q4 points at them, no scales) that
// go straight into the MFMA B operand: the same kernel without the decompression, used
// to measure what the decompression costs (W16 = false is the production kernel).
constexpr int LDS_STAGES = 3, LDS_STAGE_BYTES = BM * BK * 2;
template <bool W16>
struct LdsWeightRegs {  // int4 codes (one 16-byte load per 32 values) and raw fp16 scales
  uint4 rb[LDS_STAGES][2];
  uint32_t rsc[LDS_STAGES][2];
};
template <>
struct LdsWeightRegs<true> {  // 16-bit weights: four 16-byte loads per 32 values
  uint4 rw[LDS_STAGES][2][4];
};
//
// GATED: the gate/up product of the MLP with z = act(g) * u formed in the epilogue
// (nt_lds_store_gated); column tile t covers features 128 t .. 128 t + 127 of both segments.
template <int EPI, bool W16 = false, int NW = 8, bool GATED = false>
__global__ __launch_bounds__(64 * NW, 1) void k_gemm_nt_lds(const NtArgs a) {
  constexpr int BN = 256, WNW = 4, NJ = 2, MI = 32 / NW, NA = 32 / NW;
  // (with four waves the logits epilogue spills: measured 2.7 ms per Gemma3-4B-shaped vocabulary
  // chunk against 1.6 ms with eight)
  static_assert(NW == 8 || EPI != NT_LOGITS, "the logits epilogue takes 128-row waves");
  static_assert(!GATED || (EPI == NT_STORE_F16 && NW == 4 && !W16), "the gated epilogue is the fp16 4-wave kernel's");
  // one LDS object per ring stage, so that the compiler can tell the fragment reads of one
  // stage from the LDS-direct loads in flight into another
  __shared__ __attribute__((aligned(1024))) uint8_t lds0[LDS_STAGE_BYTES];
  __shared__ __attribute__((aligned(1024))) uint8_t lds1[LDS_STAGE_BYTES];
  __shared__ __attribute__((aligned(1024))) uint8_t lds2[LDS_STAGE_BYTES];
  // the LoRA up-projection's operands of this tile (u rows, then B rows; r <= 16 floats each),
  // copied at the start of the tile so that the epilogue does not wait for them (GATED: the
  // u rows of both segments, then the 128 B rows of each)
  __shared__ __attribute__((aligned(1024))) uint8_t lds_lora[(GATED ? 3 : 2) * BM * 16 * 4];
  auto stage_ptr = [&](auto S_) -> uint8_t* {
    constexpr int st = decltype(S_)::value;
    return st == 0 ? lds0 : st == 1 ? lds1 : lds2;
  };
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WNW, wn = wave % WNW, h = lane >> 5;
  const int nt = blockIdx.x, mt = blockIdx.y;
  int s = 0;
  if constexpr (GATED) {
    s = wn >> 1;  // waves 0, 1: gate; 2, 3: up
  } else {
    if (a.nseg > 1 && nt >= a.seg[1].tile0) s = 1;
    if (a.nseg > 2 && nt >= a.seg[2].tile0) s = 2;
  }
  const NtSeg sg = pick_seg(a, s);
  const int n0 = GATED ? nt * (BN / 2) : (nt - sg.tile0) * BN, m0 = mt * BM;
  const int K = a.K, Nn = sg.N, Kh = K >> 1;
  const int nk = (K + BK - 1) / BK, kgroups = (K + 31) >> 5;
  const int z = blockIdx.z, S = gridDim.z;
  const int kt_begin = (int)((long long)nk * z / S), kt_end = (int)((long long)nk * (z + 1) / S);

  const rsrc_t rA = make_rsrc((const u16*)a.X + (size_t)m0 * a.lda, (size_t)min(BM, a.M - m0) * a.lda * 2);
  const int wcol0 = GATED ? n0 + (wn & 1) * 32 * NJ : n0 + wn * 32 * NJ;
  const int wrows = max(0, min(32 * NJ, Nn - wcol0));
  const rsrc_t rB = W16 ? make_rsrc((const u16*)sg.q4 + (size_t)min(wcol0, Nn) * K, (size_t)wrows * K * 2)
                       : make_rsrc(sg.q4 + (size_t)min(wcol0, Nn) * Kh, (size_t)wrows * Kh);
  const rsrc_t rS = make_rsrc(W16 ? nullptr : sg.scale + (size_t)min(wcol0, Nn) * kgroups,
                              W16 ? 0 : (size_t)wrows * kgroups * 2);
  // activation loads: instruction i of wave w fills tile rows 8 (w + 8 i) .. +8, lane l row
  // 8 (w + 8 i) + l / 8, LDS position l % 8, i.e. global chunk (l % 8) ^ swz(row)
  uint32_t offA[NA];
  int chunkA[NA];
#pragma unroll
  for (int i = 0; i < NA; ++i) {
    const int row = 8 * (wave + NW * i) + (lane >> 3);
    chunkA[i] = (lane & 7) ^ ((row >> 1) & 7);
    offA[i] = (uint32_t)((row * a.lda + 8 * chunkA[i]) * 2);
  }
  const uint32_t offB = W16 ? (uint32_t)(((lane & 31) * K + 32 * h) * 2) : (uint32_t)((lane & 31) * Kh + 16 * h);
  const uint32_t offS = (uint32_t)(((lane & 31) * kgroups + h) * 2);
  // fragment reads: row wm*128 + 32 i + (l % 32), chunk 4h + t at position (4h + t) ^ swz(row)
  // with swz(row) = (row / 2) % 8 = (l / 2) % 8: the 16 lanes that read in one LDS cycle
  // (16 consecutive rows) hit 16 distinct 16-byte bank groups (rows r and r + 8 no longer
  // share one: with swz = row % 8 half of the LDS cycles were bank conflicts)
  const uint32_t rowA = (uint32_t)((wm * 32 * MI + (lane & 31)) * 128);

  LdsWeightRegs<W16> wr;
  f32x16 acc[MI][NJ];
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int j = 0; j < NJ; ++j)
#pragma unroll
      for (int q = 0; q < 16; ++q) acc[i][j][q] = 0.f;
  const bool tail = (K % BK) != 0;
  // (the rank is 8 or 16 whenever a LoRA factor is given)
  typedef __attribute__((address_space(3))) uint8_t lds_u8;
  if constexpr (GATED) {
    // per segment: BM u rows (r KiB) and the tile's 128 B rows (r / 2 KiB), 1 KiB per wave
    // and instruction
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      if (!a.seg[t].lora_B) continue;
      const rsrc_t rU = make_rsrc(a.seg[t].lora_u, (size_t)a.M * a.r * 4);
      const rsrc_t rL = make_rsrc(a.seg[t].lora_B, (size_t)a.seg[t].N * a.r * 4);
      for (int i = wave; i < a.r; i += NW)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rU, (lds_u8*)(lds_lora + t * (BM * 16 * 4) + 1024 * i), 16,
                                                 (uint32_t)(m0 * a.r * 4 + 1024 * i + 16 * lane), 0, 0, 0);
      for (int i = wave; i < a.r / 2; i += NW)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rL, (lds_u8*)(lds_lora + 2 * (BM * 16 * 4) + t * (128 * 16 * 4) + 1024 * i),
                                                 16, (uint32_t)(n0 * a.r * 4 + 1024 * i + 16 * lane), 0, 0, 0);
    }
  }
  const bool lora_lds = !GATED && EPI != NT_LOGITS && sg.lora_B;
  if (lora_lds) {
    // BM rows of r floats = r KiB each for u and B: one 1 KiB copy per wave and instruction
    // (rows past M or N read as zero)
    const int nin = a.r;
    const rsrc_t rU = make_rsrc(sg.lora_u, (size_t)a.M * a.r * 4);
    const rsrc_t rL = make_rsrc(sg.lora_B, (size_t)Nn * a.r * 4);
    for (int i = wave; i < nin; i += NW) {
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rU, (lds_u8*)(lds_lora + 1024 * i), 16,
                                               (uint32_t)(m0 * a.r * 4 + 1024 * i + 16 * lane), 0, 0, 0);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rL, (lds_u8*)(lds_lora + BM * 16 * 4 + 1024 * i), 16,
                                               (uint32_t)(n0 * a.r * 4 + 1024 * i + 16 * lane), 0, 0, 0);
    }
  }

  auto gload = [&](auto S_, int kt) {
    constexpr int st = decltype(S_)::value;  // ring stage (registers and LDS)
    const int k0 = kt * BK;
    __attribute__((address_space(3))) uint8_t* dst = (__attribute__((address_space(3))) uint8_t*)stage_ptr(S_);
#pragma unroll
    for (int i = 0; i < NA; ++i) {
      // chunks past the reduction length read as zero (out-of-range offset)
      const uint32_t off = (!tail || k0 + 8 * chunkA[i] < K) ? offA[i] + 2 * k0 : 0x80000000u;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rA, dst + 1024 * (wave + NW * i), 16, off, 0, 0, 0);
    }
    if constexpr (W16) {
#pragma unroll
      for (int j = 0; j < NJ; ++j)
#pragma unroll
        for (int t = 0; t < 4; ++t) wr.rw[st][j][t] = bload128(rB, offB + (uint32_t)((32 * j * K + k0 + 8 * t) * 2));
      if (tail && k0 + BK > K) {
        const int kb = k0 + 32 * h;
#pragma unroll
        for (int j = 0; j < NJ; ++j)
#pragma unroll
          for (int t = 0; t < 4; ++t)
            if (kb + 8 * t >= K) wr.rw[st][j][t] = make_uint4(0, 0, 0, 0);
      }
    } else {
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        wr.rb[st][j] = bload128(rB, offB + (uint32_t)(32 * j * Kh) + (k0 >> 1));
        wr.rsc[st][j] = bload16(rS, offS + (uint32_t)(32 * j * kgroups * 2) + 2 * (k0 >> 5));
      }
      if (tail && k0 + BK > K) {
        const int kb = k0 + 32 * h;
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
          if (kb >= K) wr.rsc[st][j] = 0u;
          if (kb + 0 >= K) wr.rb[st][j].x = 0u;
          if (kb + 8 >= K) wr.rb[st][j].y = 0u;
          if (kb + 16 >= K) wr.rb[st][j].z = 0u;
          if (kb + 24 >= K) wr.rb[st][j].w = 0u;
        }
      }
    }
  };
  auto mma = [&](auto S_) {
    constexpr int st = decltype(S_)::value;
    const uint8_t* As = stage_ptr(S_) + rowA;
    f16x2 sc[NJ];
    if constexpr (!W16) {
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        const _Float16 v = __builtin_bit_cast(_Float16, (uint16_t)wr.rsc[st][j]);
        sc[j] = f16x2{v, v};
      }
    }
    auto rd = [&](int t, uint4 (&dst)[MI]) {
      const int pos = ((4 * h + t) ^ ((lane >> 1) & 7)) * 16;
#pragma unroll
      for (int i = 0; i < MI; ++i) dst[i] = *(const uint4*)(As + 4096 * i + pos);
    };
    if constexpr (W16) {
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        uint4 af[MI];
        rd(t, af);
#pragma unroll
        for (int i = 0; i < MI; ++i)
#pragma unroll
          for (int j = 0; j < NJ; ++j) acc[i][j] = mfma32<OpF16>(af[i], wr.rw[st][j][t], acc[i][j]);
      }
    } else {
      // software pipeline over the four substeps: the fragments of substep t + 1 are read,
      // and its weights decompressed, while the MFMAs of substep t run (scheduling barriers
      // keep the compiler from moving the reads next to their use; the decompression is
      // interleaved one MFMA to five VALU instructions)
      uint4 af[2][MI], bq[2][NJ];
      auto dq = [&](int t, uint4 (&dst)[NJ]) {
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
          const uint32_t w = t == 0 ? wr.rb[st][j].x : t == 1 ? wr.rb[st][j].y : t == 2 ? wr.rb[st][j].z : wr.rb[st][j].w;
          dst[j] = dequant8_natural(w, sc[j]);
        }
      };
      rd(0, af[0]);
      dq(0, bq[0]);
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        if (t < 3) rd(t + 1, af[(t + 1) & 1]);
        __builtin_amdgcn_sched_barrier(0);
        if (t < 3) dq(t + 1, bq[(t + 1) & 1]);
#pragma unroll
        for (int i = 0; i < MI; ++i)
#pragma unroll
          for (int j = 0; j < NJ; ++j) acc[i][j] = mfma32<OpF16>(af[t & 1][i], bq[t & 1][j], acc[i][j]);
        if (t < 3) {
#pragma unroll
          for (int q = 0; q < MI * NJ; ++q) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
            // VALU per MFMA: five with 128-row waves, three with 256-row waves (two or four
            // measured slower)
            __builtin_amdgcn_sched_group_barrier(0x002, MI == 4 ? 5 : 3, 0);
          }
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  };
  // Step of tile k (ring stage I): issue the loads of tile k+2 into stage I+2 (last read by
  // tile k-1, before the previous barrier), the MFMAs of tile k, then wait until this
  // thread's activation loads of tile k+1 have landed (the loads issued after them: the
  // weights of k+1 and all of k+2, 2 NJ + 4 + 2 NJ) and meet the other waves at the barrier.
  // vector-memory instructions of one gload: 4 activation loads plus the weight loads
  constexpr int VMI = NA + (W16 ? 4 * NJ : 2 * NJ);
  auto step = [&](auto I_, int k) {
    constexpr int I = decltype(I_)::value;
    gload(IC<(I + 2) % LDS_STAGES>{}, min(k + 2, kt_end - 1));
    mma(IC<I>{});
    wait_vmcnt<VMI + (W16 ? 4 * NJ : 2 * NJ)>();
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");  // no LDS access moves across the barrier
  };
  if (kt_begin < kt_end) {
    gload(IC<0>{}, kt_begin);
    gload(IC<1>{}, min(kt_begin + 1, kt_end - 1));
    wait_vmcnt<VMI + (W16 ? 4 * NJ : 2 * NJ)>();  // tile kt_begin's activations (weights and tile +1 may fly)
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    int k = kt_begin;
    for (; k + 3 <= kt_end; k += 3) {
      step(IC<0>{}, k);
      step(IC<1>{}, k + 1);
      step(IC<2>{}, k + 2);
    }
    if (k < kt_end) step(IC<0>{}, k);
    if (k + 1 < kt_end) step(IC<1>{}, k + 1);
  }
  if constexpr (GATED) {
    wait_vmcnt<0>();
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    auto region = [&](int w) -> float* {
      return reinterpret_cast<float*>((w < 3 ? lds0 : lds1) + (w % 3) * (32 * 68 * 4));
    };
    const float* Us = reinterpret_cast<const float*>(lds_lora + s * (BM * 16 * 4));
    const float* Bs = reinterpret_cast<const float*>(lds_lora + 2 * (BM * 16 * 4) + s * (128 * 16 * 4));
    auto epi = [&](auto K_) {
      constexpr int KIND = decltype(K_)::value;
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        f32x16 (&ah)[4][NJ] = *reinterpret_cast<f32x16 (*)[4][NJ]>(&acc[4 * hh][0]);
        nt_lds_store_gated<KIND>(ah, a, sg, m0 + 128 * hh, wcol0, lane, region(wave), region(wave ^ 2), Us, Bs,
                                 128 * hh, (wn & 1) * 32 * NJ, s);
      }
    };
    if (a.act == 0)
      epi(IC<0>{});
    else
      epi(IC<1>{});
  } else if constexpr (EPI != NT_LOGITS) {
    // the ring is idle once the clamped loads of the last steps have landed and every wave
    // has read its last tile; each wave then stages through its own 32 x 68 fp32 region
    wait_vmcnt<0>();
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    uint8_t* reg = (wave < 3 ? lds0 : wave < 6 ? lds1 : lds2) + (wave % 3) * (32 * 68 * 4);
#pragma unroll
    for (int hh = 0; hh < MI / 4; ++hh) {
      f32x16 (&ah)[4][NJ] = *reinterpret_cast<f32x16 (*)[4][NJ]>(&acc[4 * hh][0]);
      const int r0 = wm * 32 * MI + 128 * hh;
      nt_lds_store<EPI, true>(ah, a, sg, m0 + r0, wcol0, lane, reinterpret_cast<float*>(reg),
                              reinterpret_cast<const float*>(lds_lora), r0, wn * 32 * NJ);
    }
  } else if constexpr (NW == 8) {
    // (one split: the logits GEMM runs unsplit)
    wait_vmcnt<0>();
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    uint8_t* reg = (wave < 3 ? lds0 : wave < 6 ? lds1 : lds2) + (wave % 3) * (32 * 68 * 4);
    nt_lds_logits_store(acc, a, sg, m0 + wm * 128, wcol0, lane, reinterpret_cast<float*>(reg));
  }
}

// ---------------------------------------------------------------------------- transposed
// C[m][c] = sum_seg sum_n G_seg[m][n] W_seg[n][c] (+ sum_seg du_seg A_seg), bf16 operands.
// The weight tile (64 rows n x BN columns c) is decompressed per thread as RPT rows x 16
// columns and written transposed, n-contiguous, into LDS.
// Instruction order of one K step of k_gemm_tn_big. With one wave per SIMD nothing hides
// the decompression of the next weight tile, its LDS stores or the fragment reads but the
// wave's own MFMAs, so they are spread evenly between them: the first fragment reads, then
// per MFMA four VALU instructions, one LDS store and one fragment read.
template <int NJ>
DEV void sched_tn_step() {
  __builtin_amdgcn_sched_group_barrier(0x100, 4 + NJ, 0);
#pragma unroll
  for (int i = 0; i < 16 * NJ; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x002, 4, 0);
    __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
  }
}

// The 16-bit-weight step has about a sixth of that VALU work (byte permutes instead of
// conversions): per MFMA one VALU instruction, one LDS store and one fragment read (none or
// two VALU instructions per MFMA measured 7-9 % slower).
template <int NJ>
DEV void sched_tn_step_w16() {
  __builtin_amdgcn_sched_group_barrier(0x100, 4 + NJ, 0);
#pragma unroll
  for (int i = 0; i < 16 * NJ; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x002, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
  }
}

// W16: the weights are bf16 values [N][Kout] (seg.q4 points at them, no scales), moved into
// the transposed LDS tile without decompression. The training path uses it on a transient
// copy that a decompression pass writes just before (the same operands as the int4 kernel,
// with the conversion's VALU work taken out of the main loop).
template <int BN, int EPI, bool W16 = false>
__global__ __launch_bounds__(NTH, 1) void k_gemm_tn_big(const TnArgs a) {
  constexpr int NJ = BN / 64;
  constexpr int CG = BN / 16;   // 16-column groups
  constexpr int RG = NTH / CG;  // row groups
  constexpr int RPT = BK / RG;  // weight rows per thread (4 or 2)
  __shared__ __attribute__((aligned(16))) u16 As2[2][BM * LDT];
  __shared__ __attribute__((aligned(16))) u16 Bs2[2][BN * LDT];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const TileId tl = xcd_tile();
  const int c0 = tl.x * BN, m0 = tl.y * BM;
  const int Kout = a.Kout, Kh = Kout >> 1, kgroups = (Kout + 31) >> 5;
  const int z = tl.z, S = gridDim.z;

  int ntl[3], total = 0;
#pragma unroll
  for (int s = 0; s < 3; ++s) {
    ntl[s] = s < a.nseg ? (a.seg[s].N + BK - 1) / BK : 0;
    total += ntl[s];
  }
  const int t_begin = (int)((long long)total * z / S), t_end = (int)((long long)total * (z + 1) / S);

  rsrc_t rA[3], rB[3], rS[3];
#pragma unroll
  for (int s = 0; s < 3; ++s) {
    const TnSeg& sg = a.seg[s < a.nseg ? s : 0];
    rA[s] = make_rsrc((const u16*)sg.G + (size_t)m0 * sg.ldg, (size_t)min(BM, a.M - m0) * sg.ldg * 2);
    rB[s] = W16 ? make_rsrc(sg.q4, (size_t)sg.N * Kout * 2) : make_rsrc(sg.q4, (size_t)sg.N * Kh);
    rS[s] = make_rsrc(W16 ? nullptr : sg.scale, W16 ? 0 : (size_t)sg.N * kgroups * 2);
  }
  // row group varies fastest across lanes so that the transposed LDS writes do not collide
  const int rq = tid % RG, cq = tid / RG;
  const int kc = c0 + 16 * cq;
  const uint32_t offB = W16 ? (uint32_t)((RPT * rq * Kout + kc) * 2) : (uint32_t)(RPT * rq * Kh + (kc >> 1));
  const uint32_t offS = (uint32_t)((RPT * rq * kgroups + (kc >> 5)) * 2);

  uint4 ra[2][8];
  uint2 rw[2][RPT];
  uint32_t rsc[2][RPT];
  uint4 rw16[W16 ? 2 : 1][W16 ? RPT : 1][2];  // W16: 16 bf16 weights of each row
  f32x16 acc[4][NJ];
  zero_acc(acc);

  auto locate = [&](int t, int& s, int& n0) {
    if (t < ntl[0]) {
      s = 0;
    } else if (t < ntl[0] + ntl[1]) {
      s = 1;
      t -= ntl[0];
    } else {
      s = 2;
      t -= ntl[0] + ntl[1];
    }
    n0 = t * BK;
  };

  auto run = [&](auto TAIL_) {
    constexpr bool TAIL = decltype(TAIL_)::value;
    auto gload = [&](auto S_, int t) {
      constexpr int st = decltype(S_)::value;
      int s, n0;
      locate(t, s, n0);
      const TnSeg& sg = a.seg[s];
      const rsrc_t ra_ = s == 0 ? rA[0] : s == 1 ? rA[1] : rA[2];
      const rsrc_t rb_ = s == 0 ? rB[0] : s == 1 ? rB[1] : rB[2];
      const rsrc_t rs_ = s == 0 ? rS[0] : s == 1 ? rS[1] : rS[2];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int c = tid + NTH * i;
        ra[st][i] = bload128(ra_, (uint32_t)(((c >> 3) * sg.ldg + (c & 7) * 8 + n0) * 2));
      }
#pragma unroll
      for (int i = 0; i < RPT; ++i) {
        if constexpr (W16) {
          rw16[st][i][0] = bload128(rb_, offB + (uint32_t)((n0 + i) * Kout * 2));
          rw16[st][i][1] = bload128(rb_, offB + (uint32_t)((n0 + i) * Kout * 2 + 16));
        } else {
          rw[st][i] = bload64(rb_, offB + (uint32_t)((n0 + i) * Kh));
          rsc[st][i] = bload16(rs_, offS + (uint32_t)((n0 + i) * kgroups * 2));
        }
      }
      if constexpr (TAIL) {
        if (n0 + BK > sg.N) {  // reduction tail: A columns past N must be 0 (B rows already are)
#pragma unroll
          for (int i = 0; i < 8; ++i)
            if (n0 + ((tid + NTH * i) & 7) * 8 >= sg.N) ra[st][i] = make_uint4(0, 0, 0, 0);
        }
      }
    };
    auto sstore = [&](auto S_, auto B_) {
      constexpr int st = decltype(S_)::value, bf = decltype(B_)::value;
      store_a_tile(As2[bf], tid, ra[st]);
      if constexpr (W16) {
        // bf16 weights: column e of rows i, i+1 is one 16-bit permute of their words
        uint32_t wd[RPT][8];
#pragma unroll
        for (int i = 0; i < RPT; ++i) {
          wd[i][0] = rw16[st][i][0].x; wd[i][1] = rw16[st][i][0].y; wd[i][2] = rw16[st][i][0].z;
          wd[i][3] = rw16[st][i][0].w; wd[i][4] = rw16[st][i][1].x; wd[i][5] = rw16[st][i][1].y;
          wd[i][6] = rw16[st][i][1].z; wd[i][7] = rw16[st][i][1].w;
        }
        auto pair = [&](int i, int e) {
          return (e & 1) ? perm_hi16(wd[i][e >> 1], wd[i + 1][e >> 1]) : perm_lo16(wd[i][e >> 1], wd[i + 1][e >> 1]);
        };
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          u16* dst = Bs2[bf] + (16 * cq + e) * LDT + RPT * rq;
          if constexpr (RPT == 4)
            *(uint2*)dst = make_uint2(pair(0, e), pair(2, e));
          else
            *(uint32_t*)dst = pair(0, e);
        }
      } else {
        float v[RPT][16];
#pragma unroll
        for (int i = 0; i < RPT; ++i) {
          const float sc = half_bits_to_f32((uint16_t)rsc[st][i]);
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            v[i][e] = (float)nib_s(rw[st][i].x, e) * sc;
            v[i][8 + e] = (float)nib_s(rw[st][i].y, e) * sc;
          }
        }
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          u16* dst = Bs2[bf] + (16 * cq + e) * LDT + RPT * rq;
          if constexpr (RPT == 4)
            *(uint2*)dst = make_uint2(pack_bf16x2(v[0][e], v[1][e]), pack_bf16x2(v[2][e], v[3][e]));
          else
            *(uint32_t*)dst = pack_bf16x2(v[0][e], v[1][e]);
        }
      }
    };
    auto step = [&](auto I_, int t) {
      constexpr int I = decltype(I_)::value;
      gload(IC<I>{}, min(t + 2, t_end - 1));
      mma_tile<OpBF16, NJ>(As2[I], Bs2[I], wm, wn, lane, acc);
      sstore(IC<1 - I>{}, IC<1 - I>{});
      if constexpr (W16)
        sched_tn_step_w16<NJ>();
      else
        sched_tn_step<NJ>();
      __syncthreads();
    };
    gload(IC<0>{}, t_begin);
    gload(IC<1>{}, min(t_begin + 1, t_end - 1));
    sstore(IC<0>{}, IC<0>{});
    __syncthreads();
    int t = t_begin;
    for (; t + 2 <= t_end; t += 2) {
      step(IC<0>{}, t);
      step(IC<1>{}, t + 1);
    }
    if (t < t_end) step(IC<0>{}, t);
  };
  if (t_begin < t_end) {
    bool tail = false;
    for (int s = 0; s < a.nseg; ++s) tail |= (a.seg[s].N % BK) != 0;
    if (tail)
      run(IC<1>{});
    else
      run(IC<0>{});
  }

  if constexpr (EPI == TN_PARTIAL_F32) {
    store_partial<NJ>(acc, a.out + (size_t)z * a.M * a.ldo, a.M, a.ldo, Kout - c0, m0, c0, wm, wn, lane);
    return;
  } else {
    if (S > 1) {
      store_partial<NJ>(acc, a.part + (size_t)z * a.M * Kout, a.M, Kout, Kout - c0, m0, c0, wm, wn, lane);
      return;
    }
    for (int s = 0; s < a.nseg; ++s) {
      const TnSeg& sg = a.seg[s];
      if (sg.lora_A)
        lora_mfma<NJ>(acc, sg.lora_du, a.r, m0 + wm * 128, a.M, 1.0f, sg.lora_A, 1, Kout, c0 + wn * 32 * NJ, Kout,
                      lane);
    }
    if constexpr (EPI == TN_ACT_BWD && 4 * 64 * (32 * NJ + 4) * 4 <= (int)sizeof(As2)) {
      // dz -> (dg, du) reads g, u and writes dg, du: the accumulators go through LDS so that
      // every lane handles 8 consecutive columns of a row (16-byte accesses, a wave covers
      // eight whole 128-byte row segments) instead of 2-byte accesses in the MFMA layout.
      // Each wave stages its 128 x 32NJ block in two halves of 64 rows in its own LDS region;
      // the g and u loads of a half are all issued before its accumulators are staged, so
      // their latency is paid once per half. Kout is a multiple of 32 (a group divides it).
      constexpr int CW = 32 * NJ, LDE = CW + 4, CPR = CW / 8, RPP = 64 / CPR, NP = 64 / RPP;
      float* ep = reinterpret_cast<float*>(&As2[0][0]) + wave * 64 * LDE;
      const int rr = lane / CPR, ch = lane % CPR;
      const int cbase = c0 + wn * CW + 8 * ch;
      __syncthreads();  // every wave is done with the main loop's LDS tiles
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        uint4 gw[NP], uw[NP];
#pragma unroll
        for (int p = 0; p < NP; ++p) {
          const int m = m0 + wm * 128 + 64 * hh + p * RPP + rr;
          const bool ok = m < a.M && cbase < Kout;
          const size_t idx = ok ? (size_t)m * a.ldgu + cbase : 0;
          gw[p] = ok ? *(const uint4*)((const f16*)a.g + idx) : make_uint4(0, 0, 0, 0);
          uw[p] = ok ? *(const uint4*)((const f16*)a.u + idx) : make_uint4(0, 0, 0, 0);
        }
#pragma unroll
        for (int ii = 0; ii < 2; ++ii)
#pragma unroll
          for (int q = 0; q < 16; ++q)
#pragma unroll
            for (int j = 0; j < NJ; ++j)
              ep[(32 * ii + 8 * (q >> 2) + 4 * (lane >> 5) + (q & 3)) * LDE + 32 * j + (lane & 31)] =
                  acc[2 * hh + ii][j][q];
        __syncthreads();
        // the activation kind is a template argument here, so the element loop has no branch
        // on it, and each element takes one exponential for act and act'
        auto finish = [&](auto K_) {
          constexpr int KIND = decltype(K_)::value;
#pragma unroll
          for (int p = 0; p < NP; ++p) {
            const int r = p * RPP + rr, m = m0 + wm * 128 + 64 * hh + r;
            if (m >= a.M || cbase >= Kout) continue;
            const float4 v0 = *(const float4*)(ep + r * LDE + 8 * ch), v1 = *(const float4*)(ep + r * LDE + 8 * ch + 4);
            const size_t idx = (size_t)m * a.ldgu + cbase;
            const uint32_t gq[4] = {gw[p].x, gw[p].y, gw[p].z, gw[p].w}, uq[4] = {uw[p].x, uw[p].y, uw[p].z, uw[p].w};
            const float dz[8] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w};
            uint32_t og[4], ou[4];
#pragma unroll
            for (int t = 0; t < 4; ++t) {
              const float g0 = f16_lo(gq[t]), g1 = f16_hi(gq[t]), u0 = f16_lo(uq[t]), u1 = f16_hi(uq[t]);
              float a0, d0, a1, d1;
              act_and_grad<KIND>(g0, a0, d0);
              act_and_grad<KIND>(g1, a1, d1);
              og[t] = pack_bf16x2(dz[2 * t] * u0 * d0, dz[2 * t + 1] * u1 * d1);
              ou[t] = pack_bf16x2(dz[2 * t] * a0, dz[2 * t + 1] * a1);
            }
            *(uint4*)((bf16*)a.g + idx) = make_uint4(og[0], og[1], og[2], og[3]);
            *(uint4*)((bf16*)a.u + idx) = make_uint4(ou[0], ou[1], ou[2], ou[3]);
          }
        };
        if (a.act == 0)
          finish(IC<0>{});
        else
          finish(IC<1>{});
        __syncthreads();  // before the next half overwrites the staging area
      }
      return;
    }
    auto put = [&](auto FULL_) {
      constexpr bool FULL = decltype(FULL_)::value;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        const int m = m0 + acc_row(wm, i, q, lane);
        if (!FULL && m >= a.M) continue;
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
          const int c = c0 + acc_col<NJ>(wn, j, lane);
          if (!FULL && c >= Kout) continue;
          const float v = acc[i][j][q];
          if constexpr (EPI == TN_STORE_F32) {
            a.out[(size_t)m * a.ldo + c] = v;
          } else if constexpr (EPI == TN_STORE_BF16) {
            a.outb[(size_t)m * a.ldo + c] = (bf16)v;
          } else {  // TN_ACT_BWD: v = dz; g, u (fp16) -> dg, du (bf16) in place
            const size_t idx = (size_t)m * a.ldgu + c;
            const float g = (float)((const f16*)a.g)[idx], u = (float)((const f16*)a.u)[idx];
            ((bf16*)a.g)[idx] = (bf16)(v * u * act_grad_f(g, a.act));
            ((bf16*)a.u)[idx] = (bf16)(v * act_f(g, a.act));
          }
        }
      }
    };
    if (m0 + BM <= a.M && c0 + BN <= Kout)
      put(IC<1>{});
    else
      put(IC<0>{});
  }
}


// Transposed product with both operands copied into LDS by LDS-direct loads in their stored
// layouts: the gradient tile G [256 rows m][64 n] (rows of 128 B, chunks XOR-swizzled as in
// the forward kernel) and the 16-bit weight tile W [64 rows n][256 columns c] (rows of 512 B,
// 16-byte chunk c at position c ^ (2 (n % 4) + (n / 4) % 2)). The MFMA B fragments (8
// consecutive n of one column) come from gfx950's transposing LDS read (8 bytes: in each
// group of 16 lanes, lane s points at row R0 + s / 4, columns C0 + 4 (s % 4); lane i then
// receives rows R0 .. R0 + 3 of column C0 + i). Four waves of 256 rows x 64 columns; two
// ring stages (128 KiB), the next tile's copies issued before the current tile's MFMAs.
template <int EPI>
__global__ __launch_bounds__(256, 1) void k_gemm_tn_lds(const TnArgs a) {
  constexpr int NW = 4, NJ = 2, MI = 8, BNT = 256, NA = 8, NB = 8;
  constexpr int SA = BM * BK * 2, SB = BK * BNT * 2;
  static_assert(EPI == TN_ACT_BWD || EPI == TN_STORE_BF16, "the activation-backward and bf16 epilogues");
  __shared__ __attribute__((aligned(1024))) uint8_t st0[SA + SB];
  __shared__ __attribute__((aligned(1024))) uint8_t st1[SA + SB];
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6), h = lane >> 5;
  const TileId tl = xcd_tile();
  const int c0 = tl.x * BNT, m0 = tl.y * BM;
  const int Kout = a.Kout;
  int ntl[3], total = 0;
#pragma unroll
  for (int s = 0; s < 3; ++s) {
    ntl[s] = s < a.nseg ? (a.seg[s].N + BK - 1) / BK : 0;
    total += ntl[s];
  }
  rsrc_t rA[3], rB[3];
#pragma unroll
  for (int s = 0; s < 3; ++s) {
    const TnSeg& sg = a.seg[s < a.nseg ? s : 0];
    rA[s] = make_rsrc((const u16*)sg.G + (size_t)m0 * sg.ldg, (size_t)min(BM, a.M - m0) * sg.ldg * 2);
    rB[s] = make_rsrc((const u16*)sg.q4 + c0, ((size_t)(sg.N - 1) * Kout + min(BNT, Kout - c0)) * 2);
  }
  typedef __attribute__((address_space(3))) uint8_t lds_u8;
  auto swzb = [](int r) { return 2 * (r & 3) + ((r >> 2) & 1); };
  // A copies: instruction i of the wave fills rows 8 (wave + 4 i) .. + 8
  const int rowA0 = 8 * wave + (lane >> 3), chunkA = (lane & 7) ^ ((rowA0 >> 1) & 7);
  // B copies: instruction i fills rows 2 (wave + 4 i), + 1; lane l row + l / 32, position l % 32
  int rowB[NB];
  uint32_t colB[NB];
#pragma unroll
  for (int i = 0; i < NB; ++i) {
    rowB[i] = 2 * (wave + NW * i) + (lane >> 5);
    colB[i] = (uint32_t)(8 * ((lane & 31) ^ swzb(rowB[i])) * 2);
  }
  f32x16 acc[MI][NJ];
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int j = 0; j < NJ; ++j)
#pragma unroll
      for (int q = 0; q < 16; ++q) acc[i][j][q] = 0.f;

  auto stage = [&](auto S_) -> uint8_t* { return decltype(S_)::value == 0 ? st0 : st1; };
  auto gload = [&](auto S_, int t) {
    int s = 0, tt = t;
    if (tt >= ntl[0]) {
      tt -= ntl[0];
      s = 1;
      if (tt >= ntl[1]) {
        tt -= ntl[1];
        s = 2;
      }
    }
    const TnSeg& sg = a.seg[s];
    const rsrc_t ra = s == 0 ? rA[0] : s == 1 ? rA[1] : rA[2];
    const rsrc_t rb = s == 0 ? rB[0] : s == 1 ? rB[1] : rB[2];
    const int n0 = tt * BK, Ns = sg.N, ldg = sg.ldg;
    lds_u8* dst = (lds_u8*)stage(S_);
#pragma unroll
    for (int i = 0; i < NA; ++i) {
      // reduction columns past the segment read as zero
      const int row = rowA0 + 32 * i;
      const uint32_t off = n0 + 8 * chunkA < Ns ? (uint32_t)((row * ldg + n0 + 8 * chunkA) * 2) : 0x80000000u;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, dst + 1024 * (wave + NW * i), 16, (int)off, 0, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      // rows past the segment are past the resource: zero
      const uint32_t off = (uint32_t)((n0 + rowB[i]) * Kout * 2) + colB[i];
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rb, dst + SA + 1024 * (wave + NW * i), 16, (int)off, 0, 0, 0);
    }
  };
  // fragment reads
  const uint32_t rowA = (uint32_t)((lane & 31) * 128);
  const int tg = lane >> 4, ts = lane & 15;
  typedef short v4s __attribute__((ext_vector_type(4)));
  typedef __attribute__((address_space(3))) v4s lds_v4s;
  auto mma = [&](auto S_) {
    const uint8_t* As = stage(S_) + rowA;
    const uint8_t* Bs = stage(S_) + SA;
    auto rda = [&](int t, uint4 (&dst)[MI]) {
      const int pos = ((4 * h + t) ^ ((lane >> 1) & 7)) * 16;
#pragma unroll
      for (int i = 0; i < MI; ++i) dst[i] = *(const uint4*)(As + 4096 * i + pos);
    };
    // B fragment of column block j, substep t: k = 32 h + 8 t + (0..7)
    auto rdb = [&](int t, uint4 (&dst)[NJ]) {
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        uint2 v[2];
#pragma unroll
        for (int rd = 0; rd < 2; ++rd) {
          const int r = 32 * h + 8 * t + 4 * rd + (ts >> 2);
          const int col = 64 * wave + 32 * j + 16 * (tg & 1) + 4 * (ts & 3);
          const int off = r * (BNT * 2) + (((col >> 3) ^ swzb(r)) << 4) + ((col & 7) << 1);
          v[rd] = __builtin_bit_cast(uint2, __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s*)(Bs + off)));
        }
        dst[j] = make_uint4(v[0].x, v[0].y, v[1].x, v[1].y);
      }
    };
    uint4 af[2][MI], bf[2][NJ];
    rda(0, af[0]);
    rdb(0, bf[0]);
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      if (t < 3) {
        rda(t + 1, af[(t + 1) & 1]);
        rdb(t + 1, bf[(t + 1) & 1]);
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int j = 0; j < NJ; ++j) acc[i][j] = mfma32<OpBF16>(af[t & 1][i], bf[t & 1][j], acc[i][j]);
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  auto step = [&](auto I_, int t) {
    constexpr int I = decltype(I_)::value;
    gload(IC<1 - I>{}, min(t + 1, total - 1));
    mma(IC<I>{});
    wait_vmcnt<0>();
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
  };
  gload(IC<0>{}, 0);
  wait_vmcnt<0>();
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
  int t = 0;
  for (; t + 2 <= total; t += 2) {
    step(IC<0>{}, t);
    step(IC<1>{}, t + 1);
  }
  if (t < total) step(IC<0>{}, t);

  // epilogue per 128-row half (the accumulators of rows 128 hh .. + 128 in the layout of the
  // 128-row waves of k_gemm_tn_big, with wm = hh and wn = wave)
#pragma unroll
  for (int hh = 0; hh < 2; ++hh) {
    f32x16 (&ah)[4][NJ] = *reinterpret_cast<f32x16 (*)[4][NJ]>(&acc[4 * hh][0]);
    for (int s = 0; s < a.nseg; ++s) {
      const TnSeg& sg = a.seg[s];
      if (sg.lora_A)
        lora_mfma<NJ>(ah, sg.lora_du, a.r, m0 + 128 * hh, a.M, 1.0f, sg.lora_A, 1, Kout, c0 + wave * 64, Kout, lane);
    }
    if constexpr (EPI == TN_ACT_BWD) {
      // 32-row chunks (one accumulator block each) through the wave's own 32 x 68 fp32 region:
      // each lane handles 8 consecutive columns of a row; the chunk's g and u loads are issued
      // before its accumulators are staged
      constexpr int CW = 64, LDE = CW + 4, CPR = CW / 8, RPP = 64 / CPR, NP = 32 / RPP;
      float* ep = reinterpret_cast<float*>(st0) + wave * 32 * LDE;
      const int rr = lane / CPR, ch = lane % CPR;
      const int cbase = c0 + wave * CW + 8 * ch;
#pragma unroll
      for (int h2 = 0; h2 < 4; ++h2) {
        uint4 gw[NP], uw[NP];
#pragma unroll
        for (int p = 0; p < NP; ++p) {
          const int m = m0 + 128 * hh + 32 * h2 + p * RPP + rr;
          const bool ok = m < a.M && cbase < Kout;
          const size_t idx = ok ? (size_t)m * a.ldgu + cbase : 0;
          gw[p] = ok ? *(const uint4*)((const f16*)a.g + idx) : make_uint4(0, 0, 0, 0);
          uw[p] = ok ? *(const uint4*)((const f16*)a.u + idx) : make_uint4(0, 0, 0, 0);
        }
#pragma unroll
        for (int q = 0; q < 16; ++q)
#pragma unroll
          for (int j = 0; j < NJ; ++j)
            ep[(8 * (q >> 2) + 4 * (lane >> 5) + (q & 3)) * LDE + 32 * j + (lane & 31)] = ah[h2][j][q];
        auto finish = [&](auto K_) {
          constexpr int KIND = decltype(K_)::value;
#pragma unroll
          for (int p = 0; p < NP; ++p) {
            const int r = p * RPP + rr, m = m0 + 128 * hh + 32 * h2 + r;
            const float4 v0 = *(const float4*)(ep + r * LDE + 8 * ch), v1 = *(const float4*)(ep + r * LDE + 8 * ch + 4);
            const uint32_t gq[4] = {gw[p].x, gw[p].y, gw[p].z, gw[p].w}, uq[4] = {uw[p].x, uw[p].y, uw[p].z, uw[p].w};
            const float dz[8] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w};
            uint32_t og[4], ou[4];
#pragma unroll
            for (int k = 0; k < 4; ++k) {
              const float g0 = f16_lo(gq[k]), g1 = f16_hi(gq[k]), u0 = f16_lo(uq[k]), u1 = f16_hi(uq[k]);
              float a0, d0, a1, d1;
              act_and_grad<KIND>(g0, a0, d0);
              act_and_grad<KIND>(g1, a1, d1);
              og[k] = pack_bf16x2(dz[2 * k] * u0 * d0, dz[2 * k + 1] * u1 * d1);
              ou[k] = pack_bf16x2(dz[2 * k] * a0, dz[2 * k + 1] * a1);
            }
            if (m < a.M && cbase < Kout) {
              const size_t idx = (size_t)m * a.ldgu + cbase;
              *(uint4*)((bf16*)a.g + idx) = make_uint4(og[0], og[1], og[2], og[3]);
              *(uint4*)((bf16*)a.u + idx) = make_uint4(ou[0], ou[1], ou[2], ou[3]);
            }
          }
        };
        if (a.act == 0)
          finish(IC<0>{});
        else
          finish(IC<1>{});
      }
    } else {
      auto put = [&](auto FULL_) {
        constexpr bool FULL = decltype(FULL_)::value;
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int q = 0; q < 16; ++q) {
            const int m = m0 + acc_row(hh, i, q, lane);
            if (!FULL && m >= a.M) continue;
#pragma unroll
            for (int j = 0; j < NJ; ++j) {
              const int c = c0 + acc_col<NJ>(wave, j, lane);
              if (!FULL && c >= Kout) continue;
              a.outb[(size_t)m * a.ldo + c] = (bf16)ah[i][j][q];
            }
          }
      };
      if (m0 + BM <= a.M && c0 + BNT <= Kout)
        put(IC<1>{});
      else
        put(IC<0>{});
    }
  }
}
}  // namespace

// ------------------------------------------------------------------------------ planning
static int env_big() {
  static const int v = [] {
    const char* e = getenv("MEBP_BIG_TILES");
    return e && *e ? atoi(e) : 1;
  }();
  return v;
}

GemmPlan plan_big(int M, int ntiles256, int ntiles128, int ktiles, bool logits, int max_bn) {
  GemmPlan p{0, 0, 1};
  // the LM head's GEMMs have hundreds of column tiles (the vocabulary) even for one 256-row
  // tile of tokens; the layer GEMMs need many token tiles to fill the chip
  if (!env_big() || M < (logits ? BM : 1024)) return p;
  const int mt = (M + BM - 1) / BM;
  p.big = 1;
  if (max_bn >= 256 && (logits || mt * ntiles256 >= 192)) {
    p.bn = 256;
    return p;
  }
  p.bn = 128;
  if (logits) return p;
  const int t = mt * ntiles128;
  if (t >= 160) return p;
  int s = (256 + t - 1) / t;
  const int max_s = ktiles / 4;
  if (s > max_s) s = max_s;
  if (s > 8) s = 8;
  p.splits = s < 1 ? 1 : s;
  return p;
}

static int nt_use_lds() {
  static const int v = [] {
    const char* e = getenv("MEBP_NT_LDS");
    return e && *e ? atoi(e) : 1;
  }();
  return v;
}

// fp16 / fp32 outputs as 16-byte row chunks through LDS (required by the LDS-direct kernel,
// chosen in the other one): one split, segment widths that are multiples of 8 and 16-byte
// aligned rows
static bool nt_vec_ok(const NtArgs& a, int epi, int S) {
  bool vec = S == 1;
  for (int s = 0; s < a.nseg && epi != NT_LOGITS; ++s) {
    const NtSeg& g = a.seg[s];
    const size_t esz = epi == NT_STORE_F16 ? 2 : 4;
    vec = vec && g.N % 8 == 0 && (((uintptr_t)g.out | (size_t)g.ldo * esz) & 15) == 0 &&
          (!g.resid || (((uintptr_t)g.resid | (size_t)g.ldr * 4) & 15) == 0);
  }
  return vec;
}

bool nt_gated_fused(const NtArgs& a, int epi, int bn, int S) {
  static const int on = [] {
    const char* e = getenv("MEBP_NT_GATED");
    return e && *e ? atoi(e) : 1;
  }();
  // Only where g and u are not kept (the forward pass). The recompute, which keeps them for
  // the backward, runs the plain product and the activation kernel: fused there too, the step
  // measured 494 ms against 488 ms (the epilogue's activation work then delays the backward
  // that runs beside the recompute).
  return on && !a.store_gu && a.gated && epi == NT_STORE_F16 && bn == 256 && nt_use_lds() && a.K % 8 == 0 && nt_vec_ok(a, epi, S) &&
         a.nseg == 2 && a.seg[0].N == a.seg[1].N && a.seg[0].ldo == a.seg[0].N && a.seg[1].ldo == a.seg[1].N &&
         !a.seg[0].resid && !a.seg[1].resid && !a.seg[0].rope && !a.seg[1].rope && (a.r == 8 || a.r == 16 ||
         (!a.seg[0].lora_B && !a.seg[1].lora_B)) && ((uintptr_t)a.z_out & 15) == 0;
}

hipError_t launch_gemm_nt_big(const NtArgs& a, int epi, int bn, int S, double flops, double bytes, hipStream_t st) {
  const char* name = epi == NT_STORE_F16 ? "gemm_nt_f16out" : epi == NT_STORE_F32 ? "gemm_nt_f32out" : "gemm_nt_logits";
  if (nt_gated_fused(a, epi, bn, S)) {
    // gate/up with the activation in the epilogue: one column tile per 128 features
    const dim3 gg((a.seg[0].N + 127) / 128, (a.M + BM - 1) / BM, 1);
    MEBP_TIMED(st, name, flops, bytes,
               hipLaunchKernelGGL((k_gemm_nt_lds<NT_STORE_F16, false, 4, true>), gg, dim3(256), 0, st, a));
    return hipGetLastError();
  }
  int tiles = 0;
  for (int s = 0; s < a.nseg; ++s) tiles += (a.seg[s].N + bn - 1) / bn;
  const dim3 grid(tiles, (a.M + BM - 1) / BM, S);
  NtArgs b = a;
  int t = 0;
  for (int s = 0; s < b.nseg; ++s) {
    b.seg[s].tile0 = t;
    t += (b.seg[s].N + bn - 1) / bn;
  }
#define NT_BIG(BN_, EPI_, VEC_)                                                                       \
  MEBP_TIMED(st, name, flops, bytes,                                                                  \
             hipLaunchKernelGGL((k_gemm_nt_big<BN_, BN_ / 64, EPI_, VEC_>), grid, dim3(2 * BN_), 0, st, b))
  const bool vec = nt_vec_ok(a, epi, S);
  if (bn == 256 && nt_use_lds() && a.K % 8 == 0 && (epi == NT_LOGITS || vec)) {
#define NT_LDS(EPI_, NW_) \
  MEBP_TIMED(st, name, flops, bytes, hipLaunchKernelGGL((k_gemm_nt_lds<EPI_, false, NW_>), grid, dim3(64 * NW_), 0, st, b))
    if (epi == NT_LOGITS)
      NT_LDS(NT_LOGITS, 8);
    else if (epi == NT_STORE_F16)
      NT_LDS(NT_STORE_F16, 4);
    else
      NT_LDS(NT_STORE_F32, 4);
#undef NT_LDS
  } else if (bn == 256) {
    if (epi == NT_LOGITS) {
      NT_BIG(256, NT_LOGITS, false);
    } else if (epi == NT_STORE_F16) {
      if (vec) NT_BIG(256, NT_STORE_F16, true);
      else NT_BIG(256, NT_STORE_F16, false);
    } else {
      if (vec) NT_BIG(256, NT_STORE_F32, true);
      else NT_BIG(256, NT_STORE_F32, false);
    }
  } else if (bn == 128) {
    if (epi == NT_LOGITS) {
      NT_BIG(128, NT_LOGITS, false);
    } else if (epi == NT_STORE_F16) {
      if (vec) NT_BIG(128, NT_STORE_F16, true);
      else NT_BIG(128, NT_STORE_F16, false);
    } else {
      if (vec) NT_BIG(128, NT_STORE_F32, true);
      else NT_BIG(128, NT_STORE_F32, false);
    }
  } else {
    return hipErrorInvalidValue;
  }
#undef NT_BIG
  return hipGetLastError();
}

hipError_t launch_gemm_tn_big(const TnArgs& a, int epi, int amode, int bn, int S, double flops, double bytes,
                              hipStream_t st, bool w16) {
  const dim3 grid((a.Kout + bn - 1) / bn, (a.M + BM - 1) / BM, S);
  if (amode != TN_A_BF16) return hipErrorInvalidValue;
  const char* name = epi == TN_PARTIAL_F32 ? "gemm_tn_probs_dh"
                     : epi == TN_STORE_F32  ? "gemm_tn_f32out"
                     : epi == TN_ACT_BWD    ? "gemm_tn_act_bwd"
                                            : "gemm_tn_bf16out";
#define TN_BIG(BN_, EPI_)                                                                                    \
  do {                                                                                                       \
    if (w16)                                                                                                 \
      MEBP_TIMED(st, name, flops, bytes, hipLaunchKernelGGL((k_gemm_tn_big<BN_, EPI_, true>), grid, dim3(NTH), 0, st, a)); \
    else                                                                                                     \
      MEBP_TIMED(st, name, flops, bytes, hipLaunchKernelGGL((k_gemm_tn_big<BN_, EPI_>), grid, dim3(NTH), 0, st, a));       \
  } while (0)
#define TN_BIG_EPI(BN_)                     \
  do {                                      \
    if (epi == TN_STORE_F32) {              \
      TN_BIG(BN_, TN_STORE_F32);            \
    } else if (epi == TN_ACT_BWD) {         \
      TN_BIG(BN_, TN_ACT_BWD);              \
    } else if (epi == TN_STORE_BF16) {      \
      TN_BIG(BN_, TN_STORE_BF16);           \
    } else if (epi == TN_PARTIAL_F32) {     \
      TN_BIG(BN_, TN_PARTIAL_F32);          \
    } else {                                \
      return hipErrorInvalidValue;          \
    }                                       \
  } while (0)
  // the transposed weight tile goes through LDS; 256-wide tiles would need more than the
  // 512 registers a lane has next to 256 accumulators
  if (bn != 128) return hipErrorInvalidValue;
  // the activation-backward and bf16-output products (column counts that are multiples of
  // 256 here: 10 240, 2048) on the LDS-direct kernel with 256-wide tiles; the fp32-output
  // products keep 128-wide tiles (2560 columns: 10 tiles of 256 would leave half of the last
  // round of workgroups idle)
  static const int tl = [] {
    const char* e = getenv("MEBP_TN_LDS");
    return e && *e ? atoi(e) : 1;
  }();
  if (tl && w16 && S == 1 && (epi == TN_ACT_BWD || epi == TN_STORE_BF16) && a.Kout % 8 == 0) {
    bool ok = true;
    for (int s = 0; s < a.nseg; ++s) ok = ok && a.seg[s].N % 8 == 0 && a.seg[s].ldg % 8 == 0;
    if (ok) {
      const dim3 g2((a.Kout + 255) / 256, (a.M + BM - 1) / BM, 1);
      if (epi == TN_ACT_BWD)
        MEBP_TIMED(st, name, flops, bytes, hipLaunchKernelGGL((k_gemm_tn_lds<TN_ACT_BWD>), g2, dim3(256), 0, st, a));
      else
        MEBP_TIMED(st, name, flops, bytes, hipLaunchKernelGGL((k_gemm_tn_lds<TN_STORE_BF16>), g2, dim3(256), 0, st, a));
      return hipGetLastError();
    }
  }
  TN_BIG_EPI(128);
#undef TN_BIG_EPI
#undef TN_BIG
  return hipGetLastError();
}

hipError_t launch_gemm_probe_big(int kind, const uint8_t* q4, const uint16_t* scale, int n_out, int n_in,
                                 const void* x, int M, float* out, hipStream_t st) {
  NtArgs a{};
  a.X = x; a.lda = n_in; a.M = M; a.K = n_in; a.nseg = 1;
  a.seg[0].q4 = q4; a.seg[0].scale = scale; a.seg[0].N = n_out; a.seg[0].out = out; a.seg[0].ldo = n_out;
  const int mt = (M + BM - 1) / BM;
  switch (kind) {
    case 1:  // register-staged forward, 256 x 128 tiles
      hipLaunchKernelGGL((k_gemm_nt_big<128, 2, NT_STORE_F32, true>), dim3((n_out + 127) / 128, mt, 1), dim3(256), 0,
                         st, a);
      break;
    case 2:  // register-staged forward, 256 x 256 tiles
      hipLaunchKernelGGL((k_gemm_nt_big<256, 4, NT_STORE_F32, true>), dim3((n_out + 255) / 256, mt, 1), dim3(512), 0,
                         st, a);
      break;
    case 3:  // LDS-direct forward, 256 x 256 tiles
      hipLaunchKernelGGL((k_gemm_nt_lds<NT_STORE_F32, false, 4>), dim3((n_out + 255) / 256, mt, 1), dim3(256), 0, st, a);
      break;
    case 7: {  // the transposed 256 x 128 kernel on plain bf16 weights [n_out][n_in] (seg.q4)
      TnArgs t{};
      t.M = M; t.Kout = n_in; t.nseg = 1;
      t.seg[0].G = (const bf16*)x; t.seg[0].ldg = n_out; t.seg[0].q4 = q4; t.seg[0].N = n_out;
      t.out = out; t.ldo = n_in; t.splits = 1;
      hipLaunchKernelGGL((k_gemm_tn_big<128, TN_STORE_F32, true>), dim3((n_in + 127) / 128, mt, 1), dim3(NTH), 0, st, t);
      break;
    }
    case 6:  // the LDS-direct forward kernel on plain fp16 weights [n_out][n_in] (seg.q4)
      hipLaunchKernelGGL((k_gemm_nt_lds<NT_STORE_F32, true, 4>), dim3((n_out + 255) / 256, mt, 1), dim3(256), 0, st, a);
      break;
    case 5: {  // transposed, 256 x 128 tiles
      TnArgs t{};
      t.M = M; t.Kout = n_in; t.nseg = 1;
      t.seg[0].G = (const bf16*)x; t.seg[0].ldg = n_out; t.seg[0].q4 = q4; t.seg[0].scale = scale; t.seg[0].N = n_out;
      t.out = out; t.ldo = n_in; t.splits = 1;
      hipLaunchKernelGGL((k_gemm_tn_big<128, TN_STORE_F32>), dim3((n_in + 127) / 128, mt, 1), dim3(NTH), 0, st, t);
      break;
    }
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace mebp
