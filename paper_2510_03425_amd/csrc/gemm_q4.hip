// Int4 group-dequant GEMMs on MFMA (gfx950), the lazy decompression of Algorithm 1
// fused into the matrix products of every base projection and of the tied LM head.
//
// Both orientations use one 128x128 output tile per 256-thread workgroup (2x2 waves of
// 64x64, 16x16x32 MFMA, fp32 accumulation) and a K step of 64. Activations are staged
// global -> registers -> LDS; weights are fetched as packed int4 plus one fp16 scale per
// 32-group, decompressed once per workgroup into LDS (q*s exact in fp32, then rounded to
// nearest even), and never exist as a 16-bit matrix in HBM.
//
//  * forward  ("NT"): C[m][n] = sum_k X[m][k] W[n][k]. A lane's MFMA B operand is 8
//    consecutive k of one weight row, i.e. one dword of packed codes with one scale.
//  * transposed ("TN", input gradients): C[m][c] = sum_n G[m][n] W[n][c]. The reduction
//    runs over the weight's output dim, so each thread decompresses a 4-row x 8-column
//    block and transposes it while packing, writing k-contiguous columns to LDS.
//
// Operand precision: the forward orientation multiplies activations by weights and runs
// in fp16 (v_mfma_f32_16x16x32_f16: same rate as bf16, 3 more mantissa bits, which keeps
// the 24-34 layer recompute within the parity bound); the transposed orientation
// multiplies gradients, whose magnitudes need bf16's exponent range, and runs in bf16.
//
// Split-K: when the output has too few tiles to fill the chip (few tokens), the reduction
// is split over gridDim.z workgroups per tile. Each writes its fp32 partial plane; a
// finalize kernel spread over the whole chip sums the planes in split order (so the
// result does not depend on scheduling) and applies the epilogue.
#include <stdlib.h>

#include "device_common.h"
#include "mebp_internal.h"

namespace mebp {
namespace {

constexpr int BM = 128, BN = 128, BK = 64, LDT = BK + 8;  // LDS pitch in 16-bit elements (144 B)
constexpr int NTHREADS = 256;
typedef uint16_t u16;

template <class Op>
DEV void mma_tile(const u16* As, const u16* Bs, int wm, int wn, int lane, f32x4 (&acc)[4][4]) {
#pragma unroll
  for (int ks = 0; ks < BK; ks += 32) {
    uint4 af[4], bfr[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      af[t] = *(const uint4*)(As + (wm * 64 + t * 16 + (lane & 15)) * LDT + ks + 8 * (lane >> 4));
      bfr[t] = *(const uint4*)(Bs + (wn * 64 + t * 16 + (lane & 15)) * LDT + ks + 8 * (lane >> 4));
    }
#pragma unroll
    for (int tm = 0; tm < 4; ++tm)
#pragma unroll
      for (int tn = 0; tn < 4; ++tn) acc[tm][tn] = mfma16_raw<Op>(af[tm], bfr[tn], acc[tm][tn]);
  }
}

// A-operand staging: 4 chunks of 8 elements per thread; chunk c = tid + 256 i covers row
// c>>3, columns (c&7)*8 .. +8 of the 128x64 tile.
DEV void load_a_tile(const u16* X, int lda, int M, int Kred, int m0, int k0, int tid, uint4 (&ra)[4]) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int c = tid + NTHREADS * i;
    const int m = m0 + (c >> 3), kc = k0 + (c & 7) * 8;
    ra[i] = (m < M && kc < Kred) ? *(const uint4*)(X + (size_t)m * lda + kc) : make_uint4(0, 0, 0, 0);
  }
}
DEV void store_a_tile(u16* As, int tid, const uint4 (&ra)[4]) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int c = tid + NTHREADS * i;
    *(uint4*)(As + (c >> 3) * LDT + (c & 7) * 8) = ra[i];
  }
}

DEV void zero_acc(f32x4 (&acc)[4][4]) {
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
}

template <int N>
struct IC {
  static constexpr int value = N;
};

// Split-K: store this workgroup's partial tile into the plane of its split, row-major
// [M][ldp] fp32 at column offset c0 (the finalize kernel reduces the planes in order).
DEV void store_partial(const f32x4 (&acc)[4][4], float* plane, int M, int ldp, int ncols, int m0, int c0, int wm,
                       int wn, int lane) {
#pragma unroll
  for (int tm = 0; tm < 4; ++tm)
#pragma unroll
    for (int rr = 0; rr < 4; ++rr) {
      const int m = m0 + wm * 64 + tm * 16 + 4 * (lane >> 4) + rr;
      if (m >= M) continue;
#pragma unroll
      for (int tn = 0; tn < 4; ++tn) {
        const int c = wn * 64 + tn * 16 + (lane & 15);
        if (c < ncols) plane[(size_t)m * ldp + c0 + c] = acc[tm][tn][rr];
      }
    }
}

// ------------------------------------------------------------------------------ forward
template <int EPI>
__global__ __launch_bounds__(NTHREADS, 2) void k_gemm_nt(const NtArgs a) {
  __shared__ __attribute__((aligned(16))) u16 As2[2][BM * LDT];
  __shared__ __attribute__((aligned(16))) u16 Bs2[2][BN * LDT];
  u16* As = As2[0];
  u16* Bs = Bs2[0];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int nt = blockIdx.x;
  int s = 0;
  if (a.nseg > 1 && nt >= a.seg[1].tile0) s = 1;
  if (a.nseg > 2 && nt >= a.seg[2].tile0) s = 2;
  const NtSeg& sg = a.seg[s];
  const int n0 = (nt - sg.tile0) * BN, m0 = blockIdx.y * BM;
  const int K = a.K, Nn = sg.N;
  const int nk = (K + BK - 1) / BK, kgroups = (K + 31) >> 5;
  const int z = blockIdx.z, S = gridDim.z;
  const int kt_begin = (int)((long long)nk * z / S), kt_end = (int)((long long)nk * (z + 1) / S);

  // three register stages of prefetched tiles, two LDS buffers. Loads go through buffer
  // resources based at this tile's first row: rows past M (activations) or N (weights)
  // read as 0. Only the last K tile, when K is not a multiple of BK, masks columns.
  uint4 ra[3][4];
  uint4 rb[3];
  uint32_t rsc[3];  // raw fp16 scale bits, converted when the tile is written to LDS
  const int brow = tid >> 1, bhalf = tid & 1;
  const int Kh = K >> 1;
  const rsrc_t rA = make_rsrc((const u16*)a.X + (size_t)m0 * a.lda, (size_t)min(BM, a.M - m0) * a.lda * 2);
  const int nrows = min(BN, Nn - n0);
  const rsrc_t rB = make_rsrc(sg.q4 + (size_t)n0 * Kh, (size_t)nrows * Kh);
  const rsrc_t rS = make_rsrc(sg.scale + (size_t)n0 * kgroups, (size_t)nrows * kgroups * 2);
  uint32_t offA[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int c = tid + NTHREADS * i;
    offA[i] = (uint32_t)(((c >> 3) * a.lda + (c & 7) * 8) * 2);
  }
  const uint32_t offB = (uint32_t)(brow * Kh + 16 * bhalf), offS = (uint32_t)((brow * kgroups + bhalf) * 2);

  f32x4 acc[4][4];
  zero_acc(acc);

  // TAIL: K is not a multiple of BK, so the last K tile masks the columns past K.
  auto run = [&](auto TAIL_) {
    constexpr bool TAIL = decltype(TAIL_)::value;
    auto gload = [&](auto S_, int kt) {
      constexpr int st = decltype(S_)::value;
      const int k0 = kt * BK;
#pragma unroll
      for (int i = 0; i < 4; ++i) ra[st][i] = bload128(rA, offA[i] + 2 * k0);
      rb[st] = bload128(rB, offB + (k0 >> 1));
      rsc[st] = bload16(rS, offS + 2 * (k0 >> 5));
      if constexpr (TAIL) {
        if (k0 + BK > K) {
#pragma unroll
          for (int i = 0; i < 4; ++i)
            if (((tid + NTHREADS * i) & 7) * 8 + k0 >= K) ra[st][i] = make_uint4(0, 0, 0, 0);
          const int kb = k0 + 32 * bhalf;
          if (kb >= K) rsc[st] = 0u;
          if (kb + 0 >= K) rb[st].x = 0u;
          if (kb + 8 >= K) rb[st].y = 0u;
          if (kb + 16 >= K) rb[st].z = 0u;
          if (kb + 24 >= K) rb[st].w = 0u;
        }
      }
    };
    auto sstore = [&](auto S_, auto B_) {
      constexpr int st = decltype(S_)::value, bf = decltype(B_)::value;
      store_a_tile(As2[bf], tid, ra[st]);
      const float sc = half_bits_to_f32((uint16_t)rsc[st]);
      u16* dst = Bs2[bf] + brow * LDT + 32 * bhalf;
      *(uint4*)(dst + 0) = dequant8<OpF16>(rb[st].x, sc);
      *(uint4*)(dst + 8) = dequant8<OpF16>(rb[st].y, sc);
      *(uint4*)(dst + 16) = dequant8<OpF16>(rb[st].z, sc);
      *(uint4*)(dst + 24) = dequant8<OpF16>(rb[st].w, sc);
    };
    // step for tile k (I = (k - kt_begin) % 6): prefetch tile k+3 into the register stage
    // tile k vacated (clamped to the last tile: a redundant load, no branch), multiply
    // the LDS buffer of tile k, write tile k+1 into the other buffer, one barrier. The
    // six-step body is straight-line code, so the prefetches stay in flight across it.
    auto step = [&](auto I_, int k) {
      constexpr int I = decltype(I_)::value;
      gload(IC<I % 3>{}, min(k + 3, kt_end - 1));
      mma_tile<OpF16>(As2[I % 2], Bs2[I % 2], wm, wn, lane, acc);
      sstore(IC<(I + 1) % 3>{}, IC<(I + 1) % 2>{});
      __syncthreads();
    };
    gload(IC<0>{}, kt_begin);
    gload(IC<1>{}, min(kt_begin + 1, kt_end - 1));
    gload(IC<2>{}, min(kt_begin + 2, kt_end - 1));
    sstore(IC<0>{}, IC<0>{});
    __syncthreads();
    int k = kt_begin;
    for (; k + 6 <= kt_end; k += 6) {
      step(IC<0>{}, k);
      step(IC<1>{}, k + 1);
      step(IC<2>{}, k + 2);
      step(IC<3>{}, k + 3);
      step(IC<4>{}, k + 4);
      step(IC<5>{}, k + 5);
    }
    if (k < kt_end) step(IC<0>{}, k);
    if (k + 1 < kt_end) step(IC<1>{}, k + 1);
    if (k + 2 < kt_end) step(IC<2>{}, k + 2);
    if (k + 3 < kt_end) step(IC<3>{}, k + 3);
    if (k + 4 < kt_end) step(IC<4>{}, k + 4);
  };
  if (kt_begin < kt_end) {
    if (K % BK)
      run(IC<1>{});
    else
      run(IC<0>{});
  }

  if constexpr (EPI == NT_LOGITS) {
    // per row and this wave's 64 columns (one statistics tile): max, sum of exp(v - max);
    // the logits stored relative to that max (fp16); the fp32 target logit
    _Float16* out = (_Float16*)sg.out;
    const int cw0 = n0 + wn * 64;
    const int stile = cw0 >> 6;
#pragma unroll
    for (int tm = 0; tm < 4; ++tm) {
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        const int m = m0 + wm * 64 + tm * 16 + 4 * (lane >> 4) + rr;
        float mx = -INFINITY;
#pragma unroll
        for (int tn = 0; tn < 4; ++tn) {
          const int n = cw0 + tn * 16 + (lane & 15);
          if (n < Nn) mx = fmaxf(mx, acc[tm][tn][rr]);
        }
#pragma unroll
        for (int o = 1; o < 16; o <<= 1) mx = fmaxf(mx, __shfl_xor(mx, o, 64));
        float se = 0.f;
        const int tg = m < a.M ? a.tgt[m] : -1;
#pragma unroll
        for (int tn = 0; tn < 4; ++tn) {
          const int n = cw0 + tn * 16 + (lane & 15);
          const float v = acc[tm][tn][rr];
          if (n < Nn) {
            se += __expf(v - mx);
            if (m < a.M) {
              out[(size_t)m * sg.ldo + n] = (_Float16)(v - mx);
              if (n + a.vbase == tg) a.tgt_logit[m] = v;
            }
          }
        }
#pragma unroll
        for (int o = 1; o < 16; o <<= 1) se += __shfl_xor(se, o, 64);
        if ((lane & 15) == 0 && m < a.M && cw0 < Nn) a.stats[(size_t)m * a.ntiles + stile] = make_float2(mx, se);
      }
    }
    return;
  } else {
    if (S > 1) {
      store_partial(acc, a.part + (size_t)z * a.M * a.ldp, a.M, a.ldp, Nn - n0, m0, sg.col0 + n0, wm, wn, lane);
      return;
    }
    const int r = a.r;
    const bool lora = sg.lora_B != nullptr;
    float* Us = (float*)As;  // [BM][r+1]
    float* Vs = (float*)Bs;  // [BN][r+1]
    if (lora) {
      __syncthreads();
      for (int i = tid; i < BM * r; i += NTHREADS) {
        const int m = m0 + i / r;
        Us[(i / r) * (r + 1) + i % r] = m < a.M ? a.lora_s * sg.lora_u[(size_t)m * r + i % r] : 0.f;
      }
      for (int i = tid; i < BN * r; i += NTHREADS) {
        const int n = n0 + i / r;
        Vs[(i / r) * (r + 1) + i % r] = n < Nn ? sg.lora_B[(size_t)n * r + i % r] : 0.f;
      }
      __syncthreads();
    }
#pragma unroll
    for (int tm = 0; tm < 4; ++tm) {
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        const int ml = wm * 64 + tm * 16 + 4 * (lane >> 4) + rr;
        const int m = m0 + ml;
        if (m >= a.M) continue;
#pragma unroll
        for (int tn = 0; tn < 4; ++tn) {
          const int nl = wn * 64 + tn * 16 + (lane & 15);
          const int n = n0 + nl;
          if (n >= Nn) continue;
          float v = acc[tm][tn][rr];
          if (lora) {
            float l = 0.f;
            for (int j = 0; j < r; ++j) l += Us[ml * (r + 1) + j] * Vs[nl * (r + 1) + j];
            v += l;
          }
          if (sg.resid) v += sg.resid[(size_t)m * sg.ldr + n];
          if constexpr (EPI == NT_STORE_F16)
            ((f16*)sg.out)[(size_t)m * sg.ldo + n] = (f16)v;
          else
            ((float*)sg.out)[(size_t)m * sg.ldo + n] = v;
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------- transposed
template <int EPI>
__global__ __launch_bounds__(NTHREADS, 2) void k_gemm_tn(const TnArgs a) {
  __shared__ __attribute__((aligned(16))) u16 As2[2][BM * LDT];
  __shared__ __attribute__((aligned(16))) u16 Bs2[2][BN * LDT];
  u16* As = As2[0];
  u16* Bs = Bs2[0];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int c0 = blockIdx.x * BN, m0 = blockIdx.y * BM;
  const int Kout = a.Kout, kgroups = (Kout + 31) >> 5;
  const int z = blockIdx.z, S = gridDim.z;

  int ntl[3], total = 0;
#pragma unroll
  for (int s = 0; s < 3; ++s) {
    ntl[s] = s < a.nseg ? (a.seg[s].N + BK - 1) / BK : 0;
    total += ntl[s];
  }
  const int t_begin = (int)((long long)total * z / S), t_end = (int)((long long)total * (z + 1) / S);

  // three register stages of prefetched tiles, two LDS buffers; loads through buffer
  // resources (rows past M or past a segment's N read as 0, see the forward kernel)
  uint4 ra[3][4];
  uint32_t rw[3][4];
  uint32_t rsc[3][4];  // raw fp16 scale bits
  const int rq = tid >> 4, co = tid & 15;
  const int kc = c0 + 8 * co;
  const int Kh = Kout >> 1;
  rsrc_t rA[3], rB[3], rS[3];
#pragma unroll
  for (int s = 0; s < 3; ++s) {
    const TnSeg& sg = a.seg[s < a.nseg ? s : 0];
    rA[s] = make_rsrc((const u16*)sg.G + (size_t)m0 * sg.ldg, (size_t)min(BM, a.M - m0) * sg.ldg * 2);
    rB[s] = make_rsrc(sg.q4, (size_t)sg.N * Kh);
    rS[s] = make_rsrc(sg.scale, (size_t)sg.N * kgroups * 2);
  }
  // columns past Kout read neighbouring bytes (kept inside the resource) and only feed
  // output columns that are never stored
  const uint32_t offB = (uint32_t)(4 * rq * Kh + (kc >> 1)), offS = (uint32_t)((4 * rq * kgroups + (kc >> 5)) * 2);

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
  f32x4 acc[4][4];
  zero_acc(acc);

  // TAIL: some segment's N is not a multiple of BK (its last tile masks A columns).
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
      for (int i = 0; i < 4; ++i) {
        const int c = tid + NTHREADS * i;
        ra[st][i] = bload128(ra_, (uint32_t)(((c >> 3) * sg.ldg + (c & 7) * 8 + n0) * 2));
      }
  #pragma unroll
      for (int i = 0; i < 4; ++i) {
        rw[st][i] = bload32(rb_, offB + (uint32_t)((n0 + i) * Kh));
        rsc[st][i] = bload16(rs_, offS + (uint32_t)((n0 + i) * kgroups * 2));
      }
      if constexpr (TAIL) {
        if (n0 + BK > sg.N) {  // reduction tail: A columns past N must be 0 (B rows already are)
  #pragma unroll
          for (int i = 0; i < 4; ++i)
            if (n0 + ((tid + NTHREADS * i) & 7) * 8 >= sg.N) ra[st][i] = make_uint4(0, 0, 0, 0);
        }
      }
    };
    auto sstore = [&](auto S_, auto B_) {
      constexpr int st = decltype(S_)::value, bf = decltype(B_)::value;
      store_a_tile(As2[bf], tid, ra[st]);
      float v[4][8];
  #pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float sc = half_bits_to_f32((uint16_t)rsc[st][i]);
  #pragma unroll
        for (int j = 0; j < 8; ++j) v[i][j] = (float)nib_s(rw[st][i], j) * sc;
      }
  #pragma unroll
      for (int j = 0; j < 8; ++j) {
        uint2 pk;
        pk.x = pack_bf16x2(v[0][j], v[1][j]);
        pk.y = pack_bf16x2(v[2][j], v[3][j]);
        *(uint2*)(Bs2[bf] + (8 * co + j) * LDT + 4 * rq) = pk;
      }
    };
    // same pipeline as the forward kernel
    auto step = [&](auto I_, int t) {
      constexpr int I = decltype(I_)::value;
      gload(IC<I % 3>{}, min(t + 3, t_end - 1));
      mma_tile<OpBF16>(As2[I % 2], Bs2[I % 2], wm, wn, lane, acc);
      sstore(IC<(I + 1) % 3>{}, IC<(I + 1) % 2>{});
      __syncthreads();
    };
    gload(IC<0>{}, t_begin);
    gload(IC<1>{}, min(t_begin + 1, t_end - 1));
    gload(IC<2>{}, min(t_begin + 2, t_end - 1));
    sstore(IC<0>{}, IC<0>{});
    __syncthreads();
    int t = t_begin;
    for (; t + 6 <= t_end; t += 6) {
      step(IC<0>{}, t);
      step(IC<1>{}, t + 1);
      step(IC<2>{}, t + 2);
      step(IC<3>{}, t + 3);
      step(IC<4>{}, t + 4);
      step(IC<5>{}, t + 5);
    }
    if (t < t_end) step(IC<0>{}, t);
    if (t + 1 < t_end) step(IC<1>{}, t + 1);
    if (t + 2 < t_end) step(IC<2>{}, t + 2);
    if (t + 3 < t_end) step(IC<3>{}, t + 3);
    if (t + 4 < t_end) step(IC<4>{}, t + 4);
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
    // raw partial planes, reduced by the caller
#pragma unroll
    for (int tm = 0; tm < 4; ++tm)
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        const int m = m0 + wm * 64 + tm * 16 + 4 * (lane >> 4) + rr;
        if (m >= a.M) continue;
#pragma unroll
        for (int tn = 0; tn < 4; ++tn) {
          const int c = c0 + wn * 64 + tn * 16 + (lane & 15);
          if (c < Kout) a.out[((size_t)z * a.M + m) * a.ldo + c] = acc[tm][tn][rr];
        }
      }
    return;
  } else {
    if (S > 1) {
      store_partial(acc, a.part + (size_t)z * a.M * Kout, a.M, Kout, Kout - c0, m0, c0, wm, wn, lane);
      return;
    }
    // LoRA term sum_seg du_seg[m][:] . A_seg[:][c]
    const int r = a.r;
    float* Us = (float*)As;  // [BM][r+1]
    float* Vs = (float*)Bs;  // [BN][r+1]
    for (int s = 0; s < a.nseg; ++s) {
      const TnSeg& sg = a.seg[s];
      if (sg.lora_A == nullptr) continue;
      __syncthreads();
      for (int i = tid; i < BM * r; i += NTHREADS) {
        const int m = m0 + i / r;
        Us[(i / r) * (r + 1) + i % r] = m < a.M ? sg.lora_du[(size_t)m * r + i % r] : 0.f;
      }
      for (int i = tid; i < BN * r; i += NTHREADS) {
        const int j = i / BN, c = c0 + i % BN;
        Vs[(i % BN) * (r + 1) + j] = c < Kout ? sg.lora_A[(size_t)j * Kout + c] : 0.f;
      }
      __syncthreads();
#pragma unroll
      for (int tm = 0; tm < 4; ++tm)
#pragma unroll
        for (int rr = 0; rr < 4; ++rr) {
          const int ml = wm * 64 + tm * 16 + 4 * (lane >> 4) + rr;
#pragma unroll
          for (int tn = 0; tn < 4; ++tn) {
            const int nl = wn * 64 + tn * 16 + (lane & 15);
            float l = 0.f;
            for (int j = 0; j < r; ++j) l += Us[ml * (r + 1) + j] * Vs[nl * (r + 1) + j];
            acc[tm][tn][rr] += l;
          }
        }
    }

#pragma unroll
    for (int tm = 0; tm < 4; ++tm) {
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        const int m = m0 + wm * 64 + tm * 16 + 4 * (lane >> 4) + rr;
        if (m >= a.M) continue;
#pragma unroll
        for (int tn = 0; tn < 4; ++tn) {
          const int c = c0 + wn * 64 + tn * 16 + (lane & 15);
          if (c >= Kout) continue;
          const float v = acc[tm][tn][rr];
          if constexpr (EPI == TN_STORE_F32) {
            a.out[(size_t)m * a.ldo + c] = v;
          } else if constexpr (EPI == TN_STORE_BF16) {
            a.outb[(size_t)m * a.ldo + c] = to_bf16(v);
          } else {  // TN_ACT_BWD: v = dz; reads fp16 g, u and overwrites them with bf16 dg, du
            const size_t idx = (size_t)m * a.ldgu + c;
            const float g = (float)((const f16*)a.g)[idx], u = (float)((const f16*)a.u)[idx];
            ((bf16*)a.g)[idx] = to_bf16(v * u * act_grad_f(g, a.act));
            ((bf16*)a.u)[idx] = to_bf16(v * act_f(g, a.act));
          }
        }
      }
    }
  }
}

// ------------------------------------------------------------------------ split finalize
// Sum the split planes in split order and apply the epilogue plus any fused follow-up.
// Plain mapping: one thread per 4 consecutive output columns of one row (all segment
// widths are multiples of 4).

DEV float4 sum_planes(const float* part, int S, size_t plane, size_t off) {
  // four planes in flight at a time; the sum still runs in split order
  const float* p = part + off;
  float4 v = *(const float4*)p;
  int z = 1;
  for (; z + 4 <= S; z += 4) {
    const float4 w0 = *(const float4*)(p + z * plane), w1 = *(const float4*)(p + (z + 1) * plane);
    const float4 w2 = *(const float4*)(p + (z + 2) * plane), w3 = *(const float4*)(p + (z + 3) * plane);
    v.x += w0.x; v.y += w0.y; v.z += w0.z; v.w += w0.w;
    v.x += w1.x; v.y += w1.y; v.z += w1.z; v.w += w1.w;
    v.x += w2.x; v.y += w2.y; v.z += w2.z; v.w += w2.w;
    v.x += w3.x; v.y += w3.y; v.z += w3.z; v.w += w3.w;
  }
  for (; z < S; ++z) {
    const float4 w = *(const float4*)(p + z * plane);
    v.x += w.x; v.y += w.y; v.z += w.z; v.w += w.w;
  }
  return v;
}

// sum over the 256 threads of a workgroup (every thread gets the result)
DEV float2 block_sum2(float2 v, float2* red) {
  v.x = wave_sum(v.x);
  v.y = wave_sum(v.y);
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  return make_float2(red[0].x + red[1].x + red[2].x + red[3].x, red[0].y + red[1].y + red[2].y + red[3].y);
}

// R consecutive fp32 values (16-byte aligned) into registers, all loads issued together
template <int R>
DEV void load_row(const float* p, float (&v)[R]) {
#pragma unroll
  for (int j = 0; j < R; j += 4) {
    const float4 t = *(const float4*)(p + j);
    v[j] = t.x; v[j + 1] = t.y; v[j + 2] = t.z; v[j + 3] = t.w;
  }
}

// LoRA up-projection term s * u[m] . B[n] for 4 consecutive columns n..n+3 (rank R; the
// dot product runs in rank order)
template <int R>
DEV void add_lora4_r(float (&o)[4], const float* urow, const float* B, float s, int n) {
  float u[R], b[4][R];
  load_row<R>(urow, u);
#pragma unroll
  for (int q = 0; q < 4; ++q) load_row<R>(B + (size_t)(n + q) * R, b[q]);
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    float l = 0.f;
#pragma unroll
    for (int j = 0; j < R; ++j) l += u[j] * b[q][j];
    o[q] += s * l;
  }
}
DEV void add_lora4(float (&o)[4], const NtSeg& sg, float s, int r, int m, int n) {
  if (!sg.lora_B) return;
  if (r == 8)
    add_lora4_r<8>(o, sg.lora_u + (size_t)m * 8, sg.lora_B, s, n);
  else
    add_lora4_r<16>(o, sg.lora_u + (size_t)m * 16, sg.lora_B, s, n);
}

// o[0..3] += sum_j du[m][j] * A[j][c..c+3] over the adapted segments (rank R, rank order)
template <int R>
DEV void add_lora_dx4_r(float (&o)[4], const float* durow, const float* A, int ldA, int c) {
  float du[R];
  float4 av[R];
  load_row<R>(durow, du);
#pragma unroll
  for (int j = 0; j < R; ++j) av[j] = *(const float4*)(A + (size_t)j * ldA + c);
#pragma unroll
  for (int j = 0; j < R; ++j) {
    o[0] += du[j] * av[j].x; o[1] += du[j] * av[j].y; o[2] += du[j] * av[j].z; o[3] += du[j] * av[j].w;
  }
}
DEV void add_lora_dx4(float (&o)[4], const TnArgs& a, int m, int c) {
  for (int sgi = 0; sgi < a.nseg; ++sgi) {
    const TnSeg& sg = a.seg[sgi];
    if (!sg.lora_A) continue;
    if (a.r == 8)
      add_lora_dx4_r<8>(o, sg.lora_du + (size_t)m * 8, sg.lora_A, a.Kout, c);
    else
      add_lora_dx4_r<16>(o, sg.lora_du + (size_t)m * 16, sg.lora_A, a.Kout, c);
  }
}

DEV void store4_f16(f16* p, const float (&o)[4]) {
  *(uint2*)p = make_uint2(pack_f16x2(o[0], o[1]), pack_f16x2(o[2], o[3]));
}

// Work items per row: a RoPE segment contributes one item per 4 columns of the first half
// of each head (the item also covers the partner columns dh/2 further), other segments
// one item per 4 columns.
template <int EPI>
__global__ __launch_bounds__(256) void k_nt_finalize(const NtArgs a, int S, int items) {
  const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= (size_t)a.M * items) return;
  const int m = (int)(i / items), it = (int)(i % items);
  int s = 0;
  if (a.nseg > 1 && it >= a.seg[1].item0) s = 1;
  if (a.nseg > 2 && it >= a.seg[2].item0) s = 2;
  const NtSeg& sg = a.seg[s];
  const size_t plane = (size_t)a.M * a.ldp;
  const int li = it - sg.item0;
  if (sg.rope) {
    const int dh = a.rope_dh, half = dh / 2, per_head = half / 4;
    const int n1 = (li / per_head) * dh + (li % per_head) * 4, n2 = n1 + half, e = n1 % dh;
    const float4 v1 = sum_planes(a.part, S, plane, (size_t)m * a.ldp + sg.col0 + n1);
    const float4 v2 = sum_planes(a.part, S, plane, (size_t)m * a.ldp + sg.col0 + n2);
    float o1[4] = {v1.x, v1.y, v1.z, v1.w}, o2[4] = {v2.x, v2.y, v2.z, v2.w};
    add_lora4(o1, sg, a.lora_s, a.r, m, n1);
    add_lora4(o2, sg, a.lora_s, a.r, m, n2);
    const int t = m % a.rope_T;
    float r1[4], r2[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const float2 cs = *(const float2*)(a.rope_cs + 2 * ((size_t)t * half + e + q));
      r1[q] = o1[q] * cs.x - o2[q] * cs.y;
      r2[q] = o2[q] * cs.x + o1[q] * cs.y;
    }
    store4_f16((f16*)sg.out + (size_t)m * sg.ldo + n1, r1);
    store4_f16((f16*)sg.out + (size_t)m * sg.ldo + n2, r2);
    return;
  }
  const int n = li * 4;
  const float4 v = sum_planes(a.part, S, plane, (size_t)m * a.ldp + sg.col0 + n);
  float o[4] = {v.x, v.y, v.z, v.w};
  add_lora4(o, sg, a.lora_s, a.r, m, n);
  if (sg.resid) {
    const float4 rv = *(const float4*)(sg.resid + (size_t)m * sg.ldr + n);
    o[0] += rv.x; o[1] += rv.y; o[2] += rv.z; o[3] += rv.w;
  }
  if constexpr (EPI == NT_STORE_F16)
    store4_f16((f16*)sg.out + (size_t)m * sg.ldo + n, o);
  else
    *(float4*)((float*)sg.out + (size_t)m * sg.ldo + n) = make_float4(o[0], o[1], o[2], o[3]);
}

// gate/up: z = act(g) * u for 4 columns; g, u themselves stored only when asked
__global__ __launch_bounds__(256) void k_nt_finalize_gated(const NtArgs a, int S) {
  const int c4n = a.seg[0].N >> 2;
  const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= (size_t)a.M * c4n) return;
  const int m = (int)(i / c4n), n = (int)(i % c4n) * 4;
  const size_t plane = (size_t)a.M * a.ldp;
  const NtSeg& sgg = a.seg[0];
  const NtSeg& sgu = a.seg[1];
  const float4 gv = sum_planes(a.part, S, plane, (size_t)m * a.ldp + sgg.col0 + n);
  const float4 uv = sum_planes(a.part, S, plane, (size_t)m * a.ldp + sgu.col0 + n);
  float g[4] = {gv.x, gv.y, gv.z, gv.w}, u[4] = {uv.x, uv.y, uv.z, uv.w};
  add_lora4(g, sgg, a.lora_s, a.r, m, n);
  add_lora4(u, sgu, a.lora_s, a.r, m, n);
  // the activation sees the same fp16-rounded g and u the backward will read
  float z[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    g[q] = (float)(f16)g[q];
    u[q] = (float)(f16)u[q];
    z[q] = act_f(g[q], a.act) * u[q];
  }
  if (a.store_gu) {
    store4_f16((f16*)sgg.out + (size_t)m * sgg.ldo + n, g);
    store4_f16((f16*)sgu.out + (size_t)m * sgu.ldo + n, u);
  }
  store4_f16(a.z_out + (size_t)m * a.seg[0].N + n, z);
}

// single fp32-output segment h (+ residual): also c = fp16(h * w * rstd(h)); one workgroup
// per row, each thread 4 columns out of every 1024
__global__ __launch_bounds__(256) void k_nt_finalize_norm(const NtArgs a, int S) {
  __shared__ float2 red[4];
  const int row = blockIdx.x, tid = threadIdx.x;
  const NtSeg& sg = a.seg[0];
  const int N = sg.N, c4n = N >> 2;
  const size_t plane = (size_t)a.M * a.ldp;
  constexpr int MAXC = 4;  // up to 4096 columns
  float4 h[MAXC];
  float ss = 0.f;
#pragma unroll
  for (int q = 0; q < MAXC; ++q) {
    const int c = tid + 256 * q;
    if (c < c4n) {
      const int n = c * 4;
      const float4 v = sum_planes(a.part, S, plane, (size_t)row * a.ldp + sg.col0 + n);
      float o[4] = {v.x, v.y, v.z, v.w};
      add_lora4(o, sg, a.lora_s, a.r, row, n);
      if (sg.resid) {
        const float4 rv = *(const float4*)(sg.resid + (size_t)row * sg.ldr + n);
        o[0] += rv.x; o[1] += rv.y; o[2] += rv.z; o[3] += rv.w;
      }
      h[q] = make_float4(o[0], o[1], o[2], o[3]);
      *(float4*)((float*)sg.out + (size_t)row * sg.ldo + n) = h[q];
      ss += o[0] * o[0] + o[1] * o[1] + o[2] * o[2] + o[3] * o[3];
    }
  }
  ss = block_sum2(make_float2(ss, 0.f), red).x;
  const float rs = 1.0f / sqrtf(ss / (float)N + a.eps);
#pragma unroll
  for (int q = 0; q < MAXC; ++q) {
    const int c = tid + 256 * q;
    if (c < c4n) {
      const float4 w = *(const float4*)(a.norm_w + c * 4);
      const float o[4] = {h[q].x * rs * w.x, h[q].y * rs * w.y, h[q].z * rs * w.z, h[q].w * rs * w.w};
      store4_f16(a.norm_out + (size_t)row * N + c * 4, o);
    }
  }
}

template <int EPI>
__global__ __launch_bounds__(256) void k_tn_finalize(const TnArgs a, int S) {
  const int c4n = a.Kout >> 2;
  const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= (size_t)a.M * c4n) return;
  const int m = (int)(i / c4n), c = (int)(i % c4n) * 4;
  const float4 v = sum_planes(a.part, S, (size_t)a.M * a.Kout, (size_t)m * a.Kout + c);
  float o[4] = {v.x, v.y, v.z, v.w};
  add_lora_dx4(o, a, m, c);
  if constexpr (EPI == TN_STORE_F32) {
    *(float4*)(a.out + (size_t)m * a.ldo + c) = make_float4(o[0], o[1], o[2], o[3]);
  } else if constexpr (EPI == TN_STORE_BF16) {
    const uint2 ob = make_uint2(pack_bf16x2(o[0], o[1]), pack_bf16x2(o[2], o[3]));
    *(uint2*)(a.outb + (size_t)m * a.ldo + c) = ob;
    if (a.delta) {
      // the attention backward's delta from the stored (bf16) values: the dh/4 threads of a
      // (row, head) are consecutive lanes (Kout/4 threads per row, a multiple of dh/4)
      const uint2 ov = *(const uint2*)(a.delta_o + (size_t)m * a.ldo + c);
      float acc = bf16_lo(ob.x) * f16_lo(ov.x) + bf16_hi(ob.x) * f16_hi(ov.x) + bf16_lo(ob.y) * f16_lo(ov.y) +
                  bf16_hi(ob.y) * f16_hi(ov.y);
      const int G = a.delta_dh >> 2;
      for (int k = 1; k < G; k <<= 1) acc += __shfl_xor(acc, k, 64);
      if (c % a.delta_dh == 0) {
        const int T = a.delta_T, H = a.Kout / a.delta_dh;
        const int b = m / T, t = m % T, h = c / a.delta_dh;
        a.delta[((size_t)b * H + h) * T + t] = acc;
      }
    }
  } else {  // TN_ACT_BWD
    const size_t idx = (size_t)m * a.ldgu + c;
    const uint2 gv = *(const uint2*)((const f16*)a.g + idx), uv = *(const uint2*)((const f16*)a.u + idx);
    const float g[4] = {f16_lo(gv.x), f16_hi(gv.x), f16_lo(gv.y), f16_hi(gv.y)};
    const float u[4] = {f16_lo(uv.x), f16_hi(uv.x), f16_lo(uv.y), f16_hi(uv.y)};
    float dg[4], dup[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      dg[q] = o[q] * u[q] * act_grad_f(g[q], a.act);
      dup[q] = o[q] * act_f(g[q], a.act);
    }
    *(uint2*)((bf16*)a.g + idx) = make_uint2(pack_bf16x2(dg[0], dg[1]), pack_bf16x2(dg[2], dg[3]));
    *(uint2*)((bf16*)a.u + idx) = make_uint2(pack_bf16x2(dup[0], dup[1]), pack_bf16x2(dup[2], dup[3]));
  }
}

// v (= the gradient at a norm's output) stays in registers and feeds the norm backward:
// out2 = resid2 + rstd * (w*v - xhat * mean(xhat*w*v)), xhat = x * rstd; one workgroup per row
__global__ __launch_bounds__(256) void k_tn_finalize_norm(const TnArgs a, int S) {
  __shared__ float2 red[4];
  const int row = blockIdx.x, tid = threadIdx.x;
  const int N = a.Kout, c4n = N >> 2;
  constexpr int MAXC = 4;
  float4 g[MAXC], xv[MAXC];
  float ss = 0.f, sd = 0.f;
#pragma unroll
  for (int q = 0; q < MAXC; ++q) {
    const int c = tid + 256 * q;
    if (c < c4n) {
      const int n = c * 4;
      const float4 v = sum_planes(a.part, S, (size_t)a.M * N, (size_t)row * N + n);
      float o[4] = {v.x, v.y, v.z, v.w};
      add_lora_dx4(o, a, row, n);
      g[q] = make_float4(o[0], o[1], o[2], o[3]);
      xv[q] = *(const float4*)(a.norm_x + (size_t)row * N + n);
      const float4 w = *(const float4*)(a.norm_w + n);
      ss += xv[q].x * xv[q].x + xv[q].y * xv[q].y + xv[q].z * xv[q].z + xv[q].w * xv[q].w;
      sd += xv[q].x * w.x * o[0] + xv[q].y * w.y * o[1] + xv[q].z * w.z * o[2] + xv[q].w * w.w * o[3];
    }
  }
  const float2 t = block_sum2(make_float2(ss, sd), red);
  const float rs = 1.0f / sqrtf(t.x / (float)N + a.eps);
  const float mt = rs * t.y / (float)N;
#pragma unroll
  for (int q = 0; q < MAXC; ++q) {
    const int c = tid + 256 * q;
    if (c < c4n) {
      const int n = c * 4;
      const float4 w = *(const float4*)(a.norm_w + n);
      float4 r = a.resid2 ? *(const float4*)(a.resid2 + (size_t)row * N + n) : make_float4(0.f, 0.f, 0.f, 0.f);
      r.x += rs * (w.x * g[q].x - xv[q].x * rs * mt);
      r.y += rs * (w.y * g[q].y - xv[q].y * rs * mt);
      r.z += rs * (w.z * g[q].z - xv[q].z * rs * mt);
      r.w += rs * (w.w * g[q].w - xv[q].w * rs * mt);
      *(float4*)(a.out2 + (size_t)row * N + n) = r;
      if (a.out2b)
        *(uint2*)(a.out2b + (size_t)row * N + n) = make_uint2(pack_bf16x2(r.x, r.y), pack_bf16x2(r.z, r.w));
    }
  }
}

}  // namespace

int gemm_nt_tiles(int N) { return (N + BN - 1) / BN; }

// Tuning knobs (environment, read once): MEBP_SPLIT_MAX caps the split count, MEBP_SPLIT_TARGET
// is the workgroup count the split aims for, MEBP_SPLIT_MIN_KTILES the smallest slice.
static int env_int(const char* name, int dflt) {
  const char* v = getenv(name);
  return v && *v ? atoi(v) : dflt;
}
int gemm_splits(int tiles, int ktiles) {
  static const int max_splits = env_int("MEBP_SPLIT_MAX", 16);
  static const int target = env_int("MEBP_SPLIT_TARGET", 256);
  static const int min_kt = env_int("MEBP_SPLIT_MIN_KTILES", 4);
  if (tiles >= target * 5 / 8) return 1;
  int s = (target + tiles - 1) / tiles;
  const int max_s = ktiles / (min_kt > 0 ? min_kt : 1);
  if (s > max_s) s = max_s;
  if (s > max_splits) s = max_splits;
  return s < 1 ? 1 : s;
}

size_t gemm_part_floats(int M, int ncols, int splits) { return splits > 1 ? (size_t)splits * M * ncols : 0; }

GemmPlan plan_nt(int M, const int* Ns, int nseg, int K, int epi) {
  int t256 = 0, t128 = 0;
  for (int s = 0; s < nseg; ++s) {
    t256 += (Ns[s] + 255) / 256;
    t128 += (Ns[s] + 127) / 128;
  }
  const int nk = (K + BK - 1) / BK;
  // (the logits GEMM gains from the large tiles only from two token tiles on; the dH GEMM
  // of the LM head already from one)
  if (epi == NT_LOGITS && M < 512) return GemmPlan{0, 0, 1};
  GemmPlan p = plan_big(M, t256, t128, nk, epi == NT_LOGITS, env_int("MEBP_NT_MAX_BN", 256));
  if (!p.big) p.splits = epi == NT_LOGITS ? 1 : gemm_splits(t128 * ((M + BM - 1) / BM), nk);
  return p;
}

int gemm_logit_stat_tiles(int V) { return (V + 63) / 64; }  // every kernel's waves cover 64 columns

GemmPlan plan_tn(int M, int Kout, const int* Ns, int nseg, bool softmax) {
  int kt = 0;
  for (int s = 0; s < nseg; ++s) kt += (Ns[s] + BK - 1) / BK;
  GemmPlan p = plan_big(M, (Kout + 255) / 256, (Kout + 127) / 128, kt, softmax, 128);
  if (!p.big) p.splits = gemm_splits(((Kout + BN - 1) / BN) * ((M + BM - 1) / BM), kt);
  return p;
}

hipError_t launch_gemm_nt(const NtArgs& a0, int epi, hipStream_t st, hipEvent_t lora_ready) {
  NtArgs a = a0;
  int tiles = 0, ncat = 0, items = 0;
  double flops = 0, bytes = (double)a.M * a.K * 2;
  const int kg = (a.K + 31) / 32;
  for (int s = 0; s < a.nseg; ++s) {
    a.seg[s].tile0 = tiles;
    a.seg[s].col0 = ncat;
    a.seg[s].item0 = items;
    tiles += gemm_nt_tiles(a.seg[s].N);
    ncat += a.seg[s].N;
    items += a.seg[s].rope ? a.seg[s].N / 8 : a.seg[s].N / 4;
    const double n = a.seg[s].N;
    flops += 2.0 * a.M * n * a.K;
    bytes += n * (a.K / 2 + 2 * kg) + (double)a.M * n * (epi == NT_STORE_F32 ? 4 : 2);
    if (a.seg[s].resid) bytes += (double)a.M * n * 4;
  }
  const int mt = (a.M + BM - 1) / BM;
  int Ns[3];
  for (int s = 0; s < a.nseg; ++s) Ns[s] = a.seg[s].N;
  const GemmPlan plan = plan_nt(a.M, Ns, a.nseg, a.K, epi);
  int S = plan.splits;
  if (S > 1 && (!a.part || a.part_floats < gemm_part_floats(a.M, ncat, S))) S = 1;
  if (a.norm_w && a.seg[0].N > 4096) S = 1;  // the fused row norm keeps a row in one workgroup
  a.ldp = ncat;
  dim3 grid(tiles, mt, S);
  if (lora_ready && S == 1) {
    const hipError_t ew = hipStreamWaitEvent(st, lora_ready, 0);
    if (ew != hipSuccess) return ew;
  }
  bool fused_act = false;
  if (plan.big) {
    fused_act = nt_gated_fused(a, epi, plan.bn, S);
    hipError_t eb = launch_gemm_nt_big(a, epi, plan.bn, S, flops, bytes, st);
    if (eb != hipSuccess) return eb;
  } else switch (epi) {
    case NT_STORE_F16:
      MEBP_TIMED(st, "gemm_nt_f16out", flops, bytes,
                 hipLaunchKernelGGL(k_gemm_nt<NT_STORE_F16>, grid, dim3(NTHREADS), 0, st, a));
      break;
    case NT_STORE_F32:
      MEBP_TIMED(st, "gemm_nt_f32out", flops, bytes,
                 hipLaunchKernelGGL(k_gemm_nt<NT_STORE_F32>, grid, dim3(NTHREADS), 0, st, a));
      break;
    case NT_LOGITS:
      MEBP_TIMED(st, "gemm_nt_logits", flops, bytes,
                 hipLaunchKernelGGL(k_gemm_nt<NT_LOGITS>, grid, dim3(NTHREADS), 0, st, a));
      break;
    default: return hipErrorInvalidValue;
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || epi == NT_LOGITS) return e;
  if (S == 1) {
    // unsplit: the GEMM epilogue stored the outputs; run the follow-ups as their own kernels
    for (int s = 0; s < a.nseg; ++s) {
      if (!a.seg[s].rope) continue;
      e = launch_rope_fwd((f16*)a.seg[s].out, a.seg[s].ldo, a.M / a.rope_T, a.rope_T, a.seg[s].N / a.rope_dh,
                          a.rope_dh, a.rope_cs, st);
      if (e != hipSuccess) return e;
    }
    if (a.gated && !fused_act)
      return launch_act_fwd((const f16*)a.seg[0].out, (const f16*)a.seg[1].out, a.z_out, (size_t)a.M * a.seg[0].N,
                            a.act, st);
    if (a.norm_w)
      return launch_rmsnorm_fwd((const float*)a.seg[0].out, a.norm_w, a.M, a.seg[0].N, a.eps, a.norm_out, nullptr, st);
    return hipSuccess;
  }
  const double fb = 4.0 * S * a.M * ncat + (double)a.M * ncat * (epi == NT_STORE_F16 ? 2 : 4);
  if (lora_ready && (e = hipStreamWaitEvent(st, lora_ready, 0)) != hipSuccess) return e;
  if (a.gated) {
    const size_t n = (size_t)a.M * (a.seg[0].N / 4);
    MEBP_TIMED(st, "splitk_finalize_gated", 0.0, fb,
               hipLaunchKernelGGL(k_nt_finalize_gated, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, a, S));
  } else if (a.norm_w) {
    MEBP_TIMED(st, "splitk_finalize_norm", 0.0, fb,
               hipLaunchKernelGGL(k_nt_finalize_norm, dim3((unsigned)a.M), dim3(256), 0, st, a, S));
  } else {
    const size_t n = (size_t)a.M * items;
    const dim3 fg((unsigned)((n + 255) / 256));
    if (epi == NT_STORE_F16)
      MEBP_TIMED(st, a.seg[0].rope ? "splitk_finalize_rope" : "splitk_finalize", 0.0, fb,
                 hipLaunchKernelGGL(k_nt_finalize<NT_STORE_F16>, fg, dim3(256), 0, st, a, S, items));
    else
      MEBP_TIMED(st, "splitk_finalize", 0.0, fb, hipLaunchKernelGGL(k_nt_finalize<NT_STORE_F32>, fg, dim3(256), 0, st, a, S, items));
  }
  return hipGetLastError();
}

size_t gemm_tn_w16_elems(int M, int Kout, const int* Ns, int nseg, bool softmax) {
  if (!plan_tn(M, Kout, Ns, nseg, softmax).big) return 0;
  size_t n = 0;
  for (int s = 0; s < nseg; ++s) n += (size_t)Ns[s] * Kout;
  return n;
}

hipError_t launch_gemm_tn(const TnArgs& a0, int epi, int amode, hipStream_t st, hipEvent_t lora_ready) {
  if (amode != TN_A_BF16) return hipErrorInvalidValue;
  if (a0.delta && (epi != TN_STORE_BF16 || !a0.delta_o || a0.delta_T <= 0 || a0.M % a0.delta_T ||
                   (a0.delta_dh != 64 && a0.delta_dh != 128 && a0.delta_dh != 256) || a0.Kout % a0.delta_dh))
    return hipErrorInvalidValue;
  TnArgs a = a0;
  const int ct = (a.Kout + BN - 1) / BN, mt = (a.M + BM - 1) / BM;
  double flops = 0, bytes = 0;
  const int kg = (a.Kout + 31) / 32;
  for (int s = 0; s < a.nseg; ++s) {
    const double n = a.seg[s].N;
    flops += 2.0 * a.M * n * a.Kout;
    bytes += (double)a.M * n * 2 + n * (a.Kout / 2 + 2 * kg);
  }
  int Ns[3];
  for (int s = 0; s < a.nseg; ++s) Ns[s] = a.seg[s].N;
  // (the partial-plane epilogue is the LM head's dH product, planned as such in both A modes)
  GemmPlan plan = plan_tn(a.M, a.Kout, Ns, a.nseg, epi == TN_PARTIAL_F32);
  int S;
  if (epi == TN_PARTIAL_F32) {
    S = a.splits;
  } else {
    S = plan.splits;
    if (S > 1 && (!a.part || a.part_floats < gemm_part_floats(a.M, a.Kout, S))) S = 1;
    if (a.out2 && a.Kout > 4096) S = 1;
  }
  const double outb = (double)a.M * a.Kout;
  bytes += epi == TN_STORE_BF16 ? 2 * outb : epi == TN_ACT_BWD ? 8 * outb
         : epi == TN_PARTIAL_F32 ? 4 * outb * S : 4 * outb;
  dim3 grid(ct, mt, S);
  // the large-tile kernel on a transient bf16 copy of the weights (written before the wait
  // for the LoRA projection, so the two may overlap)
  bool w16 = false;
  if (plan.big && a.w16) {
    size_t need = 0;
    for (int s = 0; s < a.nseg; ++s) need += (size_t)a.seg[s].N * a.Kout;
    if (need <= a.w16_elems) {
      size_t off = 0;
      for (int s = 0; s < a.nseg; ++s) {
        const hipError_t ed =
            launch_dequant(a.seg[s].q4, a.seg[s].scale, a.seg[s].N, a.Kout, 32, nullptr, a.w16 + off, st);
        if (ed != hipSuccess) return ed;
        a.seg[s].q4 = reinterpret_cast<const uint8_t*>(a.w16 + off);
        a.seg[s].scale = nullptr;
        off += (size_t)a.seg[s].N * a.Kout;
      }
      w16 = true;
    }
  }
  if (lora_ready && S == 1) {
    const hipError_t ew = hipStreamWaitEvent(st, lora_ready, 0);
    if (ew != hipSuccess) return ew;
  }
  if (plan.big) {
    hipError_t eb = launch_gemm_tn_big(a, epi, amode, plan.bn, S, flops, bytes, st, w16);
    if (eb != hipSuccess) return eb;
  } else {
    switch (epi) {
      case TN_STORE_F32:
        MEBP_TIMED(st, "gemm_tn_f32out", flops, bytes,
                   hipLaunchKernelGGL((k_gemm_tn<TN_STORE_F32>), grid, dim3(NTHREADS), 0, st, a));
        break;
      case TN_ACT_BWD:
        MEBP_TIMED(st, "gemm_tn_act_bwd", flops, bytes,
                   hipLaunchKernelGGL((k_gemm_tn<TN_ACT_BWD>), grid, dim3(NTHREADS), 0, st, a));
        break;
      case TN_STORE_BF16:
        MEBP_TIMED(st, "gemm_tn_bf16out", flops, bytes,
                   hipLaunchKernelGGL((k_gemm_tn<TN_STORE_BF16>), grid, dim3(NTHREADS), 0, st, a));
        break;
      case TN_PARTIAL_F32:
        MEBP_TIMED(st, "gemm_tn_probs_dh", flops, bytes,
                   hipLaunchKernelGGL((k_gemm_tn<TN_PARTIAL_F32>), grid, dim3(NTHREADS), 0, st, a));
        break;
      default: return hipErrorInvalidValue;
    }
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || epi == TN_PARTIAL_F32) return e;
  const bool norm = epi == TN_STORE_F32 && a.out2;
  if (S == 1) {
    if (norm) return launch_rmsnorm_bwd(a.norm_x, a.norm_w, a.out, a.resid2, a.M, a.Kout, a.eps, a.out2, a.out2b, st);
    if (epi == TN_STORE_BF16 && a.delta)
      return launch_attn_delta(a.outb, a.delta_o, a.ldo, a.M / a.delta_T, a.delta_T, a.Kout / a.delta_dh, a.delta_dh,
                               a.delta, st);
    return hipSuccess;
  }
  const double fb = 4.0 * S * a.M * a.Kout + outb * (epi == TN_ACT_BWD ? 8 : epi == TN_STORE_BF16 ? 2 : 4);
  if (lora_ready && (e = hipStreamWaitEvent(st, lora_ready, 0)) != hipSuccess) return e;
  if (norm) {
    MEBP_TIMED(st, "splitk_finalize_normbwd", 0.0, fb + 16 * outb,
               hipLaunchKernelGGL(k_tn_finalize_norm, dim3((unsigned)a.M), dim3(256), 0, st, a, S));
    return hipGetLastError();
  }
  const size_t nthr = (size_t)a.M * (a.Kout / 4);
  const dim3 fg((unsigned)((nthr + 255) / 256));
  switch (epi) {
    case TN_STORE_F32:
      MEBP_TIMED(st, "splitk_finalize", 0.0, fb, hipLaunchKernelGGL(k_tn_finalize<TN_STORE_F32>, fg, dim3(256), 0, st, a, S));
      break;
    case TN_ACT_BWD:
      MEBP_TIMED(st, "splitk_finalize_actbwd", 0.0, fb, hipLaunchKernelGGL(k_tn_finalize<TN_ACT_BWD>, fg, dim3(256), 0, st, a, S));
      break;
    default:
      MEBP_TIMED(st, "splitk_finalize", 0.0, fb, hipLaunchKernelGGL(k_tn_finalize<TN_STORE_BF16>, fg, dim3(256), 0, st, a, S));
      break;
  }
  return hipGetLastError();
}

hipError_t launch_gemm_probe(int kind, const uint8_t* q4, const uint16_t* scale, int n_out, int n_in, const void* x,
                             int M, float* out, hipStream_t st) {
  if (kind == 0) {
    NtArgs a{};
    a.X = x; a.lda = n_in; a.M = M; a.K = n_in; a.nseg = 1;
    a.seg[0].q4 = q4; a.seg[0].scale = scale; a.seg[0].N = n_out; a.seg[0].out = out; a.seg[0].ldo = n_out;
    const dim3 grid(gemm_nt_tiles(n_out), (M + BM - 1) / BM, 1);
    hipLaunchKernelGGL(k_gemm_nt<NT_STORE_F32>, grid, dim3(NTHREADS), 0, st, a);
    return hipGetLastError();
  }
  if (kind == 4) {
    TnArgs a{};
    a.M = M; a.Kout = n_in; a.nseg = 1;
    a.seg[0].G = (const bf16*)x; a.seg[0].ldg = n_out; a.seg[0].q4 = q4; a.seg[0].scale = scale; a.seg[0].N = n_out;
    a.out = out; a.ldo = n_in; a.splits = 1;
    const dim3 grid((n_in + BN - 1) / BN, (M + BM - 1) / BM, 1);
    hipLaunchKernelGGL((k_gemm_tn<TN_STORE_F32>), grid, dim3(NTHREADS), 0, st, a);
    return hipGetLastError();
  }
  return launch_gemm_probe_big(kind, q4, scale, n_out, n_in, x, M, out, st);
}

}  // namespace mebp
