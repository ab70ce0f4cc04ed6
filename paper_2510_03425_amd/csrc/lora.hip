// Rank-r LoRA products on MFMA (gfx950): the adapter's down-projection u = X A^T, the
// gradient projection du = s dY B (both "rows": r <= 16 outputs per token, reduction over
// the model dimension), and the weight gradients dB = s dY^T u, dA = du^T X ("outer":
// reduction over tokens).
//
// The 16-bit activation / gradient operand is used as stored; the fp32 adapter weights
// (A, B) and fp32 u / du enter the MFMA as a hi + lo pair of 16-bit values (two MFMAs),
// which keeps their operand rounding near 2^-17 instead of 2^-9.
//
// Both kernels split their reduction across workgroups when one workgroup per output
// block would leave the chip idle; partials are summed in split order by the last
// workgroup to arrive (one atomic counter per output block), so results are deterministic.
#include "device_common.h"
#include "mebp_internal.h"

namespace mebp {
namespace {

typedef uint16_t u16;

template <class Op>
DEV void split_hi_lo(const float (&f)[8], uint4& hi, uint4& lo) {
  uint32_t h[4], l[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    h[i] = Op::pack(f[2 * i], f[2 * i + 1]);
    l[i] = Op::pack(f[2 * i] - Op::lo(h[i]), f[2 * i + 1] - Op::hi(h[i]));
  }
  hi = make_uint4(h[0], h[1], h[2], h[3]);
  lo = make_uint4(l[0], l[1], l[2], l[3]);
}

// ------------------------------------------------------------------------------ rows
// out[m][j] = s * sum_k X[m][k] W(j,k); workgroup = 64 rows x 16 outputs, 4 waves split the
// workgroup's k range; blockIdx.y splits k across workgroups.
constexpr int LR_ROWS = 64;
template <class Op>
__global__ __launch_bounds__(256) void k_lora_rows(const u16* X, int ldx, int M, int K, const float* W, int wt, int r,
                                                   float s, float* out, float* part, int* counters) {
  __shared__ float red[4][LR_ROWS][17];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int m0 = blockIdx.x * LR_ROWS, ks = blockIdx.y, KS = gridDim.y;
  const int nsteps = (K + 31) / 32;
  const int sb = (int)((long long)nsteps * ks / KS), se = (int)((long long)nsteps * (ks + 1) / KS);
  const int j = lane & 15;
  f32x4 acc[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int st = sb + w; st < se; st += 4) {
    const int k = st * 32 + 8 * (lane >> 4);
    const bool kok = k < K;
    float f[8];
    if (kok && j < r) {
      if (wt == 0) {
        const float4 a = *(const float4*)(W + (size_t)j * K + k), b = *(const float4*)(W + (size_t)j * K + k + 4);
        f[0] = a.x; f[1] = a.y; f[2] = a.z; f[3] = a.w; f[4] = b.x; f[5] = b.y; f[6] = b.z; f[7] = b.w;
      } else {
#pragma unroll
        for (int i = 0; i < 8; ++i) f[i] = W[(size_t)(k + i) * r + j];
      }
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i) f[i] = 0.f;
    }
    uint4 bh, bl;
    split_hi_lo<Op>(f, bh, bl);
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int m = m0 + t * 16 + (lane & 15);
      const uint4 av = (kok && m < M) ? *(const uint4*)(X + (size_t)m * ldx + k) : make_uint4(0, 0, 0, 0);
      acc[t] = mfma16_raw<Op>(av, bh, acc[t]);
      acc[t] = mfma16_raw<Op>(av, bl, acc[t]);
    }
  }
  // lane holds rows t*16 + 4g + rr, column j
#pragma unroll
  for (int t = 0; t < 4; ++t)
#pragma unroll
    for (int rr = 0; rr < 4; ++rr) red[w][t * 16 + 4 * (lane >> 4) + rr][j] = acc[t][rr];
  __syncthreads();
  // 64 rows x 16 columns = 1024 outputs, 4 per thread
  float v[4];
  int mm[4], jj[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int o = tid + 256 * q;
    mm[q] = o >> 4;
    jj[q] = o & 15;
    v[q] = (red[0][mm[q]][jj[q]] + red[1][mm[q]][jj[q]]) + (red[2][mm[q]][jj[q]] + red[3][mm[q]][jj[q]]);
  }
  if (KS > 1) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int m = m0 + mm[q];
      if (m < M && jj[q] < r) st_dev(&part[((size_t)ks * M + m) * r + jj[q]], v[q]);
    }
    if (!arrive_last(counters + blockIdx.x, KS)) return;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int m = m0 + mm[q];
      if (m >= M || jj[q] >= r) continue;
      float a = 0.f;
      for (int z = 0; z < KS; ++z) a += ld_dev(&part[((size_t)z * M + m) * r + jj[q]]);
      v[q] = a;
    }
  }
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int m = m0 + mm[q];
    if (m < M && jj[q] < r) out[(size_t)m * r + jj[q]] = s * v[q];
  }
}

// ----------------------------------------------------------------------------- outer
// R(c, j) = s * sum_m Mx[m][c] V[m][j]; workgroup = 128 columns c x 16 j (each wave 32 c);
// per iteration 64 tokens are staged transposed in LDS (c-major, token-contiguous) together
// with V^T as hi/lo planes; blockIdx.y splits the tokens across workgroups. The products
// run in bf16 (V may be a tiny gradient); an fp16 Mx is converted to bf16 while staged.
constexpr int LO_C = 128, LO_M = 64, LO_LD = LO_M + 8;
template <bool MX_F16>
__global__ __launch_bounds__(256) void k_lora_outer(const u16* Mx, int ldm, int M, int C, const float* V, int r,
                                                    float s, float* out, int layout, float* part, int* counters) {
  __shared__ __attribute__((aligned(16))) u16 Mt[LO_C * LO_LD];
  __shared__ __attribute__((aligned(16))) u16 Vh[16 * LO_LD];
  __shared__ __attribute__((aligned(16))) u16 Vl[16 * LO_LD];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int c0 = blockIdx.x * LO_C, ms = blockIdx.y, MS = gridDim.y;
  const int nsteps = (M + LO_M - 1) / LO_M;
  const int sb = (int)((long long)nsteps * ms / MS), se = (int)((long long)nsteps * (ms + 1) / MS);
  f32x4 acc[2] = {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}};
  for (int st = sb; st < se; ++st) {
    const int mb = st * LO_M;
    if (tid < 128) {
      // one 8x8 block of Mx (8 tokens x 8 columns) per thread, transposed into Mt[c][m]
      const int rb = tid & 7, cb = tid >> 3;  // 8 token blocks x 16 column blocks
      uint32_t in[8][4];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int m = mb + rb * 8 + i, c = c0 + cb * 8;
        uint4 v = make_uint4(0, 0, 0, 0);
        if (m < M && c < C) v = *(const uint4*)(Mx + (size_t)m * ldm + c);
        if (MX_F16) v = f16x8_to_bf16x8(v);
        in[i][0] = v.x; in[i][1] = v.y; in[i][2] = v.z; in[i][3] = v.w;
      }
#pragma unroll
      for (int jc = 0; jc < 8; ++jc) {
        uint4 o;
        if (jc & 1) {
          o = make_uint4(perm_hi16(in[0][jc >> 1], in[1][jc >> 1]), perm_hi16(in[2][jc >> 1], in[3][jc >> 1]),
                         perm_hi16(in[4][jc >> 1], in[5][jc >> 1]), perm_hi16(in[6][jc >> 1], in[7][jc >> 1]));
        } else {
          o = make_uint4(perm_lo16(in[0][jc >> 1], in[1][jc >> 1]), perm_lo16(in[2][jc >> 1], in[3][jc >> 1]),
                         perm_lo16(in[4][jc >> 1], in[5][jc >> 1]), perm_lo16(in[6][jc >> 1], in[7][jc >> 1]));
        }
        *(uint4*)(Mt + (cb * 8 + jc) * LO_LD + rb * 8) = o;
      }
    } else {
      // V^T hi/lo planes: 16 j x 64 tokens, 8 tokens per thread
      const int t = tid - 128, jv = t & 15, mq = t >> 4;  // mq: 8 token groups of 8
      float f[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int m = mb + mq * 8 + i;
        f[i] = (m < M && jv < r) ? V[(size_t)m * r + jv] : 0.f;
      }
      uint4 hi, lo;
      split_hi_lo<OpBF16>(f, hi, lo);
      *(uint4*)(Vh + jv * LO_LD + mq * 8) = hi;
      *(uint4*)(Vl + jv * LO_LD + mq * 8) = lo;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < LO_M; kk += 32) {
      const uint4 bh = *(const uint4*)(Vh + (lane & 15) * LO_LD + kk + 8 * (lane >> 4));
      const uint4 bl = *(const uint4*)(Vl + (lane & 15) * LO_LD + kk + 8 * (lane >> 4));
#pragma unroll
      for (int ct = 0; ct < 2; ++ct) {
        const uint4 av = *(const uint4*)(Mt + (w * 32 + ct * 16 + (lane & 15)) * LO_LD + kk + 8 * (lane >> 4));
        acc[ct] = mfma16_raw<OpBF16>(av, bh, acc[ct]);
        acc[ct] = mfma16_raw<OpBF16>(av, bl, acc[ct]);
      }
    }
    __syncthreads();
  }
  // lane holds R rows c = c0 + w*32 + ct*16 + 4g + rr, column j = lane%16
  const int j = lane & 15;
  if (MS > 1) {
#pragma unroll
    for (int ct = 0; ct < 2; ++ct)
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        const int c = c0 + w * 32 + ct * 16 + 4 * (lane >> 4) + rr;
        if (c < C && j < r) st_dev(&part[((size_t)ms * C + c) * r + j], acc[ct][rr]);
      }
    if (!arrive_last(counters + blockIdx.x, MS)) return;
#pragma unroll
    for (int ct = 0; ct < 2; ++ct)
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        const int c = c0 + w * 32 + ct * 16 + 4 * (lane >> 4) + rr;
        float a = 0.f;
        if (c < C && j < r)
          for (int z = 0; z < MS; ++z) a += ld_dev(&part[((size_t)z * C + c) * r + j]);
        acc[ct][rr] = a;
      }
  }
#pragma unroll
  for (int ct = 0; ct < 2; ++ct)
#pragma unroll
    for (int rr = 0; rr < 4; ++rr) {
      const int c = c0 + w * 32 + ct * 16 + 4 * (lane >> 4) + rr;
      if (c < C && j < r) out[layout == 0 ? (size_t)c * r + j : (size_t)j * C + c] = s * acc[ct][rr];
    }
}

__global__ void k_fill_i32(int* p, int n, int v) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

int rows_splits(int M, int K) {
  const int mb = (M + LR_ROWS - 1) / LR_ROWS, steps = (K + 31) / 32;
  int s = (256 + mb - 1) / mb;
  if (s > steps / 4) s = steps / 4;
  if (s > 64) s = 64;
  return s < 1 ? 1 : s;
}
int outer_splits(int M, int C) {
  const int cb = (C + LO_C - 1) / LO_C, steps = (M + LO_M - 1) / LO_M;
  int s = (256 + cb - 1) / cb;
  if (s > steps / 2) s = steps / 2;
  if (s > 64) s = 64;
  return s < 1 ? 1 : s;
}

}  // namespace

size_t lora_rows_part_floats(int M, int K, int r) {
  const int s = rows_splits(M, K);
  return s > 1 ? (size_t)s * M * r : 0;
}
size_t lora_outer_part_floats(int M, int C, int r) {
  const int s = outer_splits(M, C);
  return s > 1 ? (size_t)s * C * r : 0;
}

hipError_t launch_lora_rows(const void* X, int xbf16, int ldx, int M, int K, const float* W, int wt, int r, float s,
                            float* out, const SplitScratch& sc, hipStream_t st) {
  const int mb = (M + LR_ROWS - 1) / LR_ROWS;
  int KS = rows_splits(M, K);
  if (KS > 1 && (!sc.part || sc.part_floats < (size_t)KS * M * r || mb > sc.ncounters)) KS = 1;
  dim3 grid(mb, KS);
  const double flops = 2.0 * M * K * r, bytes = (double)M * K * 2 + (double)K * r * 4 + (double)M * r * 4;
  if (xbf16)
    MEBP_TIMED(st, "lora_rows", flops, bytes,
               hipLaunchKernelGGL(k_lora_rows<OpBF16>, grid, dim3(256), 0, st, (const u16*)X, ldx, M, K, W, wt, r, s,
                                  out, sc.part, sc.counters));
  else
    MEBP_TIMED(st, "lora_rows", flops, bytes,
               hipLaunchKernelGGL(k_lora_rows<OpF16>, grid, dim3(256), 0, st, (const u16*)X, ldx, M, K, W, wt, r, s,
                                  out, sc.part, sc.counters));
  return hipGetLastError();
}

hipError_t launch_lora_outer(const void* Mx, int mbf16, int ldm, int M, int C, const float* V, int r, float s,
                             float* out, int layout, const SplitScratch& sc, hipStream_t st) {
  const int cb = (C + LO_C - 1) / LO_C;
  int MS = outer_splits(M, C);
  if (MS > 1 && (!sc.part || sc.part_floats < (size_t)MS * C * r || cb > sc.ncounters)) MS = 1;
  dim3 grid(cb, MS);
  const double flops = 2.0 * M * C * r, bytes = (double)M * C * 2 + (double)M * r * 4 + (double)C * r * 4;
  if (mbf16)
    MEBP_TIMED(st, "lora_outer", flops, bytes,
               hipLaunchKernelGGL(k_lora_outer<false>, grid, dim3(256), 0, st, (const u16*)Mx, ldm, M, C, V, r, s, out,
                                  layout, sc.part, sc.counters));
  else
    MEBP_TIMED(st, "lora_outer", flops, bytes,
               hipLaunchKernelGGL(k_lora_outer<true>, grid, dim3(256), 0, st, (const u16*)Mx, ldm, M, C, V, r, s, out,
                                  layout, sc.part, sc.counters));
  return hipGetLastError();
}

hipError_t launch_fill_i32(int* p, int n, int v, hipStream_t st) {
  hipLaunchKernelGGL(k_fill_i32, dim3((n + 255) / 256), dim3(256), 0, st, p, n, v);
  return hipGetLastError();
}

}  // namespace mebp
