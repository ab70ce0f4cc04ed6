// Int4 group-dequant GEMMs on bf16 MFMA (gfx950), the lazy decompression of Algorithm 1
// fused into the matrix products of every base projection and of the tied LM head.
//
// Both orientations use one 128x128 output tile per 256-thread workgroup (2x2 waves of
// 64x64, 16x16x32 MFMA, fp32 accumulation) and a K step of 64. Activations are staged
// global -> registers -> LDS; weights are fetched as packed int4 plus one fp16 scale per
// 32-group, decompressed once per workgroup into LDS (q*s exact in fp32, then rounded to
// nearest even), and never exist as a 16-bit matrix in HBM.
//
// Operand precision: the forward orientation multiplies activations by weights and runs
// in fp16 (v_mfma_f32_16x16x32_f16: same rate as bf16, 3 more mantissa bits, which keeps
// the 24-34 layer recompute within the parity bound); the transposed orientation
// multiplies gradients, whose magnitudes need bf16's exponent range, and runs in bf16.
//
//  * forward  ("NT"): C[m][n] = sum_k X[m][k] W[n][k]. A lane's MFMA B operand is 8
//    consecutive k of one weight row, i.e. one dword of packed codes with one scale.
//  * transposed ("TN", input gradients): C[m][c] = sum_n G[m][n] W[n][c]. The reduction
//    runs over the weight's output dim, so each thread decompresses a 4-row x 8-column
//    block and transposes it while packing, writing k-contiguous columns to LDS.
#include "device_common.h"
#include "mebp_internal.h"

namespace mebp {
namespace {

constexpr int BM = 128, BN = 128, BK = 64, LDT = BK + 8;  // LDS pitch in bf16 (144 B)
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

// A-operand staging: 4 chunks of 8 bf16 per thread; chunk c = tid + 256 i covers row c>>3,
// columns (c&7)*8 .. +8 of the 128x64 tile.
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

// ------------------------------------------------------------------------------ forward
template <int EPI>
__global__ __launch_bounds__(NTHREADS, 2) void k_gemm_nt(const NtArgs a) {
  __shared__ __attribute__((aligned(16))) u16 As[BM * LDT];
  __shared__ __attribute__((aligned(16))) u16 Bs[BN * LDT];
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

  uint4 ra[4];
  uint32_t rb[4];
  float rsc;
  const int brow = tid >> 1, bhalf = tid & 1, bn = n0 + brow;
  const uint8_t* wrow = sg.q4 + (size_t)bn * (K >> 1);

  auto gload = [&](int kt) {
    const int k0 = kt * BK;
    load_a_tile((const u16*)a.X, a.lda, a.M, K, m0, k0, tid, ra);
    const int kb = k0 + 32 * bhalf;
    if (bn < Nn && kb < K) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int kk = kb + 8 * j;
        rb[j] = kk < K ? *(const uint32_t*)(wrow + (kk >> 1)) : 0u;
      }
      rsc = half_bits_to_f32(sg.scale[(size_t)bn * kgroups + (kb >> 5)]);
    } else {
      rb[0] = rb[1] = rb[2] = rb[3] = 0u;
      rsc = 0.f;
    }
  };
  auto sstore = [&]() {
    store_a_tile(As, tid, ra);
#pragma unroll
    for (int j = 0; j < 4; ++j) *(uint4*)(Bs + brow * LDT + 32 * bhalf + 8 * j) = dequant8<OpF16>(rb[j], rsc);
  };

  f32x4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  gload(0);
  sstore();
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    if (kt + 1 < nk) gload(kt + 1);
    mma_tile<OpF16>(As, Bs, wm, wn, lane, acc);
    __syncthreads();
    if (kt + 1 < nk) {
      sstore();
      __syncthreads();
    }
  }

  if constexpr (EPI == NT_LOGITS) {
    // fp16 logits, per-row partial (max, sum exp) over this 128-column tile, target logit
    float* red = (float*)As;  // [2 waves along n][BM] max, then sum
    _Float16* out = (_Float16*)sg.out;
#pragma unroll
    for (int tm = 0; tm < 4; ++tm) {
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        const int ml = wm * 64 + tm * 16 + 4 * (lane >> 4) + rr;
        const int m = m0 + ml;
        float mx = -INFINITY;
#pragma unroll
        for (int tn = 0; tn < 4; ++tn) {
          const int n = n0 + wn * 64 + tn * 16 + (lane & 15);
          if (n < Nn) mx = fmaxf(mx, acc[tm][tn][rr]);
        }
#pragma unroll
        for (int o = 1; o < 16; o <<= 1) mx = fmaxf(mx, __shfl_xor(mx, o, 64));
        float se = 0.f;
        const int tg = m < a.M ? a.tgt[m] : -1;
#pragma unroll
        for (int tn = 0; tn < 4; ++tn) {
          const int n = n0 + wn * 64 + tn * 16 + (lane & 15);
          const float v = acc[tm][tn][rr];
          if (n < Nn) {
            se += __expf(v - mx);
            if (m < a.M) out[(size_t)m * sg.ldo + n] = (_Float16)v;
            if (n == tg) a.tgt_logit[m] = v;
          }
        }
#pragma unroll
        for (int o = 1; o < 16; o <<= 1) se += __shfl_xor(se, o, 64);
        if ((lane & 15) == 0) {
          red[wn * BM + ml] = mx;
          red[2 * BM + wn * BM + ml] = se;
        }
      }
    }
    __syncthreads();
    if (tid < BM && m0 + tid < a.M) {
      const float m1 = red[tid], m2 = red[BM + tid];
      const float mx = fmaxf(m1, m2);
      const float se = red[2 * BM + tid] * __expf(m1 - mx) + red[3 * BM + tid] * __expf(m2 - mx);
      a.stats[(size_t)(m0 + tid) * a.ntiles + nt] = make_float2(mx, se);
    }
    return;
  } else {
    const int r = a.r;
    const bool lora = sg.lora_B != nullptr;
    float* Us = (float*)As;  // [BM][r+1]
    float* Vs = (float*)Bs;  // [BN][r+1]
    if (lora) {
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
template <int EPI, int AMODE>
__global__ __launch_bounds__(NTHREADS, 2) void k_gemm_tn(const TnArgs a) {
  __shared__ __attribute__((aligned(16))) u16 As[BM * LDT];
  __shared__ __attribute__((aligned(16))) u16 Bs[BN * LDT];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int c0 = blockIdx.x * BN, m0 = blockIdx.y * BM;
  const int Kout = a.Kout, kgroups = (Kout + 31) >> 5;

  int ntl[3], total = 0;
#pragma unroll
  for (int s = 0; s < 3; ++s) {
    ntl[s] = s < a.nseg ? (a.seg[s].N + BK - 1) / BK : 0;
    total += ntl[s];
  }
  int t_begin = 0, t_end = total;
  if (EPI == TN_PARTIAL_F32) {
    t_begin = (int)((long long)total * blockIdx.z / a.splits);
    t_end = (int)((long long)total * (blockIdx.z + 1) / a.splits);
  }

  // softmax-mode row data (rows fixed per thread for the 4 A chunks)
  float rlse[4];
  bool rval[4];
  if constexpr (AMODE == TN_A_SOFTMAX) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int m = m0 + ((tid + NTHREADS * i) >> 3);
      rval[i] = m < a.M && a.tgt[m] >= 0;
      rlse[i] = rval[i] ? a.lse[m] : 0.f;
    }
  }

  uint4 ra[4];
  uint32_t rw[4];
  float rsc[4];
  const int rq = tid >> 4, co = tid & 15;
  const int kc = c0 + 8 * co;
  int cur_n0 = 0, cur_N = 0;  // reduction offset / length of the tile held in ra

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
  auto gload = [&](int t) {
    int s, n0;
    locate(t, s, n0);
    const TnSeg& sg = a.seg[s];
    cur_n0 = n0;
    cur_N = sg.N;
    load_a_tile((const u16*)sg.G, sg.ldg, a.M, sg.N, m0, n0, tid, ra);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int n = n0 + 4 * rq + i;
      const bool ok = n < sg.N && kc < Kout;
      rw[i] = ok ? *(const uint32_t*)(sg.q4 + (size_t)n * (Kout >> 1) + (kc >> 1)) : 0u;
      rsc[i] = ok ? half_bits_to_f32(sg.scale[(size_t)n * kgroups + (kc >> 5)]) : 0.f;
    }
  };
  auto sstore = [&]() {
    if constexpr (AMODE == TN_A_SOFTMAX) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int c = tid + NTHREADS * i;
        uint4 p = make_uint4(0, 0, 0, 0);
        // chunks past the reduction length were zero-filled; they must stay 0, not exp(-lse)
        if (rval[i] && cur_n0 + (c & 7) * 8 < cur_N) {
          const uint32_t* h = (const uint32_t*)&ra[i];
          uint32_t o[4];
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const float lo = (float)__builtin_bit_cast(_Float16, (uint16_t)(h[j] & 0xffff));
            const float hi = (float)__builtin_bit_cast(_Float16, (uint16_t)(h[j] >> 16));
            o[j] = pack_bf16x2(__expf(lo - rlse[i]), __expf(hi - rlse[i]));
          }
          p = make_uint4(o[0], o[1], o[2], o[3]);
        }
        *(uint4*)(As + (c >> 3) * LDT + (c & 7) * 8) = p;
      }
    } else {
      store_a_tile(As, tid, ra);
    }
    float v[4][8];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 8; ++j) v[i][j] = (float)nib_s(rw[i], j) * rsc[i];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      uint2 pk;
      pk.x = pack_bf16x2(v[0][j], v[1][j]);
      pk.y = pack_bf16x2(v[2][j], v[3][j]);
      *(uint2*)(Bs + (8 * co + j) * LDT + 4 * rq) = pk;
    }
  };

  f32x4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  if (t_begin < t_end) {
    gload(t_begin);
    sstore();
    __syncthreads();
    for (int t = t_begin; t < t_end; ++t) {
      if (t + 1 < t_end) gload(t + 1);
      mma_tile<OpBF16>(As, Bs, wm, wn, lane, acc);
      __syncthreads();
      if (t + 1 < t_end) {
        sstore();
        __syncthreads();
      }
    }
  }

  // LoRA term sum_seg du_seg[m][:] . A_seg[:][c] (split 0 only when split)
  const int r = a.r;
  const bool add_lora = (EPI != TN_PARTIAL_F32) || blockIdx.z == 0;
  float* Us = (float*)As;  // [BM][r+1]
  float* Vs = (float*)Bs;  // [BN][r+1]
  for (int s = 0; s < a.nseg; ++s) {
    const TnSeg& sg = a.seg[s];
    if (!add_lora || sg.lora_A == nullptr) continue;
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
    __syncthreads();
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
        } else if constexpr (EPI == TN_PARTIAL_F32) {
          a.out[((size_t)blockIdx.z * a.M + m) * a.ldo + c] = v;
        } else {  // TN_ACT_BWD: v = dz
          const size_t idx = (size_t)m * a.ldgu + c;
          // reads fp16 g, u; overwrites them in place with bf16 dg, du
          const float g = (float)((const f16*)a.g)[idx], u = (float)((const f16*)a.u)[idx];
          ((bf16*)a.g)[idx] = to_bf16(v * u * act_grad_f(g, a.act));
          ((bf16*)a.u)[idx] = to_bf16(v * act_f(g, a.act));
        }
      }
    }
  }
}

}  // namespace

int gemm_nt_tiles(int N) { return (N + BN - 1) / BN; }

hipError_t launch_gemm_nt(const NtArgs& a, int epi, hipStream_t st) {
  int tiles = 0;
  for (int s = 0; s < a.nseg; ++s) tiles += gemm_nt_tiles(a.seg[s].N);
  dim3 grid(tiles, (a.M + BM - 1) / BM);
  switch (epi) {
    case NT_STORE_F16: hipLaunchKernelGGL(k_gemm_nt<NT_STORE_F16>, grid, dim3(NTHREADS), 0, st, a); break;
    case NT_STORE_F32: hipLaunchKernelGGL(k_gemm_nt<NT_STORE_F32>, grid, dim3(NTHREADS), 0, st, a); break;
    case NT_LOGITS: hipLaunchKernelGGL(k_gemm_nt<NT_LOGITS>, grid, dim3(NTHREADS), 0, st, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_gemm_tn(const TnArgs& a, int epi, int amode, hipStream_t st) {
  dim3 grid((a.Kout + BN - 1) / BN, (a.M + BM - 1) / BM, epi == TN_PARTIAL_F32 ? a.splits : 1);
  if (amode == TN_A_SOFTMAX) {
    if (epi != TN_PARTIAL_F32) return hipErrorInvalidValue;
    hipLaunchKernelGGL((k_gemm_tn<TN_PARTIAL_F32, TN_A_SOFTMAX>), grid, dim3(NTHREADS), 0, st, a);
  } else {
    switch (epi) {
      case TN_STORE_F32: hipLaunchKernelGGL((k_gemm_tn<TN_STORE_F32, TN_A_BF16>), grid, dim3(NTHREADS), 0, st, a); break;
      case TN_ACT_BWD: hipLaunchKernelGGL((k_gemm_tn<TN_ACT_BWD, TN_A_BF16>), grid, dim3(NTHREADS), 0, st, a); break;
      case TN_PARTIAL_F32: hipLaunchKernelGGL((k_gemm_tn<TN_PARTIAL_F32, TN_A_BF16>), grid, dim3(NTHREADS), 0, st, a); break;
      case TN_STORE_BF16: hipLaunchKernelGGL((k_gemm_tn<TN_STORE_BF16, TN_A_BF16>), grid, dim3(NTHREADS), 0, st, a); break;
      default: return hipErrorInvalidValue;
    }
  }
  return hipGetLastError();
}

}  // namespace mebp
