// Rank-r LoRA products on MFMA (gfx950): the adapter's down-projection u = X A^T, the
// gradient projection du = s dY B (both "rows": r <= 16 outputs per token, reduction over
// the model dimension), and the weight gradients dB = s dY^T u, dA = du^T X ("outer":
// reduction over tokens). Up to three projections that share a stage of the layer (q, k,
// v; gate, up) run in one launch (blockIdx.y selects the projection).
//
// The 16-bit activation / gradient operand is used as stored; the fp32 adapter weights
// (A, B) and fp32 u / du enter the MFMA as a hi + lo pair of 16-bit values (two MFMAs),
// which keeps their operand rounding near 2^-17 instead of 2^-9.
//
// "rows" keeps the whole reduction inside one workgroup (its waves split K, partial
// tiles summed through LDS in wave order). "outer" splits the token range over
// blockIdx.z when there are many tokens; the split partials are then summed in split
// order by a small reduce kernel. Both are deterministic.
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
// out[m][j] = s * sum_k X[m][k] W(j,k); workgroup = 64 rows x 16 outputs and LR_WAVES waves
// that take interleaved 64-wide K super-steps (every row segment a lane group loads is 128
// contiguous bytes), two super-steps in flight per iteration (one with three jobs); the
// per-wave partial tiles are summed through LDS in wave order. The many waves keep enough
// loads in flight to stream X near the HBM rate even with few row blocks.
// NJ = 1: blockIdx.y selects the job. NJ > 1: the NJ jobs share X (the q, k, v or gate, up
// down-projections of one normalised input), read once for all of them.
constexpr int LR_ROWS = 64, LR_WAVES = 8;
template <class Op, int NJ>
__global__ __launch_bounds__(64 * LR_WAVES) void k_lora_rows(const LoraRowsArgs a) {
  __shared__ float red[LR_WAVES][LR_ROWS][17];
  const int jb0 = NJ > 1 ? 0 : blockIdx.y;
  const LoraRowsJob& jx = a.job[jb0];
  const u16* X = (const u16*)jx.X;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int m0 = blockIdx.x * LR_ROWS, M = a.M, K = jx.K, r = a.r;
  const int nsup = (K + 63) / 64;
  const int j = lane & 15;

  auto load_w = [&](const float* W, int k, uint4& bh, uint4& bl) {
    float f[8];
    if (k < K && j < r) {
      if (a.wt == 0) {
        const float4 p = *(const float4*)(W + (size_t)j * K + k), q = *(const float4*)(W + (size_t)j * K + k + 4);
        f[0] = p.x; f[1] = p.y; f[2] = p.z; f[3] = p.w; f[4] = q.x; f[5] = q.y; f[6] = q.z; f[7] = q.w;
      } else {
#pragma unroll
        for (int i = 0; i < 8; ++i) f[i] = W[(size_t)(k + i) * r + j];
      }
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i) f[i] = 0.f;
    }
    split_hi_lo<Op>(f, bh, bl);
  };
  // the super-step's two 32-wide halves of rows t*16 + lane%16 (K is a multiple of 8, so a
  // chunk is either wholly inside the row or wholly past it)
  auto load_x = [&](int k, uint4 (&xv)[2][4]) {
#pragma unroll
    for (int hh = 0; hh < 2; ++hh)
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int m = m0 + t * 16 + (lane & 15), kk = k + 32 * hh;
        xv[hh][t] = (kk < K && m < M) ? *(const uint4*)(X + (size_t)m * jx.ldx + kk) : make_uint4(0, 0, 0, 0);
      }
  };
  auto mma = [&](int k, const uint4 (&xv)[2][4], f32x4 (&acc)[NJ][4]) {
#pragma unroll
    for (int q = 0; q < NJ; ++q)
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        uint4 bh, bl;
        load_w(a.job[jb0 + q].W, k + 32 * hh, bh, bl);
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          acc[q][t] = mfma16_raw<Op>(xv[hh][t], bh, acc[q][t]);
          acc[q][t] = mfma16_raw<Op>(xv[hh][t], bl, acc[q][t]);
        }
      }
  };

  f32x4 acc[NJ][4];
#pragma unroll
  for (int q = 0; q < NJ; ++q)
#pragma unroll
    for (int t = 0; t < 4; ++t) acc[q][t] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int ko = 8 * (lane >> 4);
  if constexpr (NJ < 3) {
    for (int ss = w; ss < nsup; ss += 2 * LR_WAVES) {
      const int k0 = ss * 64 + ko, k1 = (ss + LR_WAVES) * 64 + ko;
      uint4 x0[2][4], x1[2][4];
      load_x(k0, x0);
      load_x(k1, x1);
      mma(k0, x0, acc);
      mma(k1, x1, acc);
    }
  } else {
    // three jobs' accumulators leave registers for one super-step in flight
    for (int ss = w; ss < nsup; ss += LR_WAVES) {
      const int k0 = ss * 64 + ko;
      uint4 x0[2][4];
      load_x(k0, x0);
      mma(k0, x0, acc);
    }
  }
  // lane holds rows t*16 + 4g + rr, column j; one job at a time through the LDS tile
#pragma unroll
  for (int q = 0; q < NJ; ++q) {
    if (q) __syncthreads();  // the previous job's sums have been read
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) red[w][t * 16 + 4 * (lane >> 4) + rr][j] = acc[q][t][rr];
    __syncthreads();
    float* out = a.job[jb0 + q].out;
    for (int o = tid; o < LR_ROWS * 16; o += 64 * LR_WAVES) {
      const int mm = o >> 4, jj = o & 15, m = m0 + mm;
      if (m < M && jj < r) {
        float v = 0.f;
#pragma unroll
        for (int ww = 0; ww < LR_WAVES; ++ww) v += red[ww][mm][jj];
        out[(size_t)m * r + jj] = a.s * v;
      }
    }
  }
}

// ----------------------------------------------------------------------------- outer
// R(c, j) = s * sum_m Mx[m][c] V[m][j]; workgroup = 128 columns c x 16 j (each wave 32 c);
// per iteration 64 tokens are staged transposed in LDS (c-major, token-contiguous) together
// with V^T as hi/lo planes. The products run in bf16 (V may be a tiny gradient); an fp16 Mx
// is converted to bf16 while staged. The LDS tiles are double-buffered and the next
// iteration's tokens are loaded into registers while the current ones are multiplied, so
// one barrier per iteration suffices and loads overlap.
// NJ = 1: blockIdx.y selects the job. NJ > 1: the NJ jobs share Mx (dA of q, k, v or of
// gate, up: one layer input against each projection's du), staged once for all of them.
constexpr int LO_C = 128, LO_M = 64, LO_LD = LO_M + 8;
template <bool MX_F16, int NJ>
__global__ __launch_bounds__(256) void k_lora_outer(const LoraOuterArgs a) {
  __shared__ __attribute__((aligned(16))) u16 Mt[2][LO_C * LO_LD];
  __shared__ __attribute__((aligned(16))) u16 Vh[2][NJ][16 * LO_LD];
  __shared__ __attribute__((aligned(16))) u16 Vl[2][NJ][16 * LO_LD];
  const int jb0 = NJ > 1 ? 0 : blockIdx.y;
  const LoraOuterJob& jx = a.job[jb0];
  const u16* Mx = (const u16*)jx.Mx;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int C = jx.C, M = a.M, r = a.r;
  const int c0 = blockIdx.x * LO_C, ms = blockIdx.z, MS = gridDim.z;
  if (c0 >= C) return;
  const int nsteps = (M + LO_M - 1) / LO_M;
  const int sb = (int)((long long)nsteps * ms / MS), se = (int)((long long)nsteps * (ms + 1) / MS);
  // threads 0..127: one 8x8 block of Mx (8 tokens x 8 columns); 128..255: 8 tokens of V
  const bool mx_role = tid < 128;
  const int rb = tid & 7, cb = (tid >> 3) & 15;      // Mx role: token block, column block
  const int jv = (tid - 128) & 15, mq = (tid - 128) >> 4;  // V role: output j, token group
  uint32_t in[8][4];
  float f[NJ][8];
  auto load = [&](int st) {
    const int mb = st * LO_M;
    if (mx_role) {
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int m = mb + rb * 8 + i, c = c0 + cb * 8;
        uint4 v = make_uint4(0, 0, 0, 0);
        if (m < M && c < C) v = *(const uint4*)(Mx + (size_t)m * jx.ldm + c);
        in[i][0] = v.x; in[i][1] = v.y; in[i][2] = v.z; in[i][3] = v.w;
      }
    } else {
#pragma unroll
      for (int q = 0; q < NJ; ++q)
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const int m = mb + mq * 8 + i;
          f[q][i] = (m < M && jv < r) ? a.job[jb0 + q].V[(size_t)m * r + jv] : 0.f;
        }
    }
  };
  auto store = [&](int buf) {
    if (mx_role) {
      if (MX_F16) {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const uint4 v = f16x8_to_bf16x8(make_uint4(in[i][0], in[i][1], in[i][2], in[i][3]));
          in[i][0] = v.x; in[i][1] = v.y; in[i][2] = v.z; in[i][3] = v.w;
        }
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
        *(uint4*)(Mt[buf] + (cb * 8 + jc) * LO_LD + rb * 8) = o;
      }
    } else {
#pragma unroll
      for (int q = 0; q < NJ; ++q) {
        uint4 hi, lo;
        split_hi_lo<OpBF16>(f[q], hi, lo);
        *(uint4*)(Vh[buf][q] + jv * LO_LD + mq * 8) = hi;
        *(uint4*)(Vl[buf][q] + jv * LO_LD + mq * 8) = lo;
      }
    }
  };
  f32x4 acc[NJ][2];
#pragma unroll
  for (int q = 0; q < NJ; ++q) acc[q][0] = acc[q][1] = f32x4{0.f, 0.f, 0.f, 0.f};
  if (sb < se) load(sb);
  for (int st = sb; st < se; ++st) {
    const int buf = (st - sb) & 1;
    store(buf);
    __syncthreads();
    if (st + 1 < se) load(st + 1);
#pragma unroll
    for (int kk = 0; kk < LO_M; kk += 32) {
      uint4 av[2];
#pragma unroll
      for (int ct = 0; ct < 2; ++ct)
        av[ct] = *(const uint4*)(Mt[buf] + (w * 32 + ct * 16 + (lane & 15)) * LO_LD + kk + 8 * (lane >> 4));
#pragma unroll
      for (int q = 0; q < NJ; ++q) {
        const uint4 bh = *(const uint4*)(Vh[buf][q] + (lane & 15) * LO_LD + kk + 8 * (lane >> 4));
        const uint4 bl = *(const uint4*)(Vl[buf][q] + (lane & 15) * LO_LD + kk + 8 * (lane >> 4));
#pragma unroll
        for (int ct = 0; ct < 2; ++ct) {
          acc[q][ct] = mfma16_raw<OpBF16>(av[ct], bh, acc[q][ct]);
          acc[q][ct] = mfma16_raw<OpBF16>(av[ct], bl, acc[q][ct]);
        }
      }
    }
  }
  // lane holds R rows c = c0 + w*32 + ct*16 + 4g + rr, column j = lane%16
  const int j = lane & 15;
#pragma unroll
  for (int q = 0; q < NJ; ++q) {
    const LoraOuterJob& jb = a.job[jb0 + q];
    const int y = jb0 + q;
#pragma unroll
    for (int ct = 0; ct < 2; ++ct)
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        const int c = c0 + w * 32 + ct * 16 + 4 * (lane >> 4) + rr;
        if (c >= C || j >= r) continue;
        if (MS > 1)
          a.part[(((size_t)y * MS + ms) * a.cmax + c) * r + j] = acc[q][ct][rr];
        else
          jb.out[a.layout == 0 ? (size_t)c * r + j : (size_t)j * C + c] = jb.s * acc[q][ct][rr];
      }
  }
}

// sum the token-split partials of every job in split order and write with layout / scale
__global__ void k_lora_outer_reduce(const LoraOuterArgs a, int MS) {
  const LoraOuterJob& jb = a.job[blockIdx.y];
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  const int r = a.r;
  if (i >= jb.C * r) return;
  const int c = i / r, j = i % r;
  float acc = 0.f;
  for (int z = 0; z < MS; ++z) acc += a.part[(((size_t)blockIdx.y * MS + z) * a.cmax + c) * r + j];
  jb.out[a.layout == 0 ? (size_t)c * r + j : (size_t)j * jb.C + c] = jb.s * acc;
}

__global__ void k_fill_i32(int* p, int n, int v) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

// token splits of an outer launch with `groups` workgroup columns per split (column blocks
// times the jobs that do not share their input): about 512 workgroups, two per CU (LDS and
// registers allow two or three), so that one workgroup's loads overlap another's transposes
// and MFMAs (256 workgroups measured 25-35 % slower on the large launches)
int outer_splits(int M, int cmax, int groups) {
  const int cb = ((cmax + LO_C - 1) / LO_C) * groups, steps = (M + LO_M - 1) / LO_M;
  if (steps < 16) return 1;
  int s = (512 + cb - 1) / cb;
  if (s > steps / 4) s = steps / 4;
  if (s > 64) s = 64;
  return s < 1 ? 1 : s;
}

// jobs that read the same input (pointer, leading dimension and width) run in one workgroup
template <class J>
bool same_input(const J* job, int n, const void* J::*x, int J::*ld, int J::*w) {
  for (int i = 1; i < n; ++i)
    if (job[i].*x != job[0].*x || job[i].*ld != job[0].*ld || job[i].*w != job[0].*w) return false;
  return n > 1;
}

}  // namespace

size_t lora_outer_part_floats(int M, int cmax, int r, int njobs) {
  // the most splits any grouping of the jobs uses (one workgroup column group per split)
  const int s = outer_splits(M, cmax, 1);
  return s > 1 ? (size_t)njobs * s * cmax * r : 0;
}

hipError_t launch_lora_rows(const LoraRowsArgs& a, int xbf16, hipStream_t st) {
  const bool shared = same_input(a.job, a.njobs, &LoraRowsJob::X, &LoraRowsJob::ldx, &LoraRowsJob::K);
  dim3 grid((a.M + LR_ROWS - 1) / LR_ROWS, shared ? 1 : a.njobs);
  double flops = 0, bytes = 0;
  for (int i = 0; i < a.njobs; ++i) {
    flops += 2.0 * a.M * a.job[i].K * a.r;
    bytes += (i == 0 || !shared ? (double)a.M * a.job[i].K * 2 : 0.0) + (double)a.job[i].K * a.r * 4 +
             (double)a.M * a.r * 4;
  }
  const dim3 blk(64 * LR_WAVES);
#define LR_GO(OP, NJ) MEBP_TIMED(st, "lora_rows", flops, bytes, hipLaunchKernelGGL((k_lora_rows<OP, NJ>), grid, blk, 0, st, a))
  const int nj = shared ? a.njobs : 1;
  if (xbf16) {
    if (nj == 3) LR_GO(OpBF16, 3); else if (nj == 2) LR_GO(OpBF16, 2); else LR_GO(OpBF16, 1);
  } else {
    if (nj == 3) LR_GO(OpF16, 3); else if (nj == 2) LR_GO(OpF16, 2); else LR_GO(OpF16, 1);
  }
#undef LR_GO
  return hipGetLastError();
}

hipError_t launch_lora_outer(const LoraOuterArgs& a0, int mbf16, hipStream_t st) {
  LoraOuterArgs a = a0;
  const bool shared = same_input(a.job, a.njobs, &LoraOuterJob::Mx, &LoraOuterJob::ldm, &LoraOuterJob::C);
  a.cmax = 0;
  double flops = 0, bytes = 0;
  for (int i = 0; i < a.njobs; ++i) {
    a.cmax = a.job[i].C > a.cmax ? a.job[i].C : a.cmax;
    flops += 2.0 * a.M * a.job[i].C * a.r;
    bytes += (i == 0 || !shared ? (double)a.M * a.job[i].C * 2 : 0.0) + (double)a.M * a.r * 4 +
             (double)a.job[i].C * a.r * 4;
  }
  const int groups = shared ? 1 : a.njobs;
  int MS = outer_splits(a.M, a.cmax, groups);
  if (MS > 1 && (!a.part || a.part_floats < (size_t)a.njobs * MS * a.cmax * a.r)) MS = 1;
  dim3 grid((a.cmax + LO_C - 1) / LO_C, groups, MS);
  const int nj = shared ? a.njobs : 1;
#define LO_GO(F16, NJ) MEBP_TIMED(st, "lora_outer", flops, bytes, hipLaunchKernelGGL((k_lora_outer<F16, NJ>), grid, dim3(256), 0, st, a))
  if (mbf16) {
    if (nj == 3) LO_GO(false, 3); else if (nj == 2) LO_GO(false, 2); else LO_GO(false, 1);
  } else {
    if (nj == 3) LO_GO(true, 3); else if (nj == 2) LO_GO(true, 2); else LO_GO(true, 1);
  }
#undef LO_GO
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || MS == 1) return e;
  dim3 rg((a.cmax * a.r + 255) / 256, a.njobs);
  MEBP_TIMED(st, "lora_outer_reduce", 0.0, 4.0 * MS * a.cmax * a.r * a.njobs,
             hipLaunchKernelGGL(k_lora_outer_reduce, rg, dim3(256), 0, st, a, MS));
  return hipGetLastError();
}

hipError_t launch_fill_i32(int* p, int n, int v, hipStream_t st) {
  hipLaunchKernelGGL(k_fill_i32, dim3((n + 255) / 256), dim3(256), 0, st, p, n, v);
  return hipGetLastError();
}

}  // namespace mebp
