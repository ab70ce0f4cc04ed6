// Memory-bound kernels of the checkpointed LoRA step on gfx950: decompression and
// embedding gather, RMSNorm forward/backward, RoPE, gated activation, the rank-r LoRA
// projections and weight gradients, and the cross-entropy reductions of the final block.
// All reductions run in a fixed order (no atomics), so results are bit-reproducible.
#include "device_common.h"
#include "mebp_internal.h"

namespace mebp {
namespace {

// ------------------------------------------------------------------ decompression
// out[r][c] = q[r][c] * s[r][c/group]; one thread per 8 codes (one dword).
__global__ void k_dequant(const uint8_t* q4, const uint16_t* scale, int rows, int cols, int group,
                          float* out_f32, uint16_t* out_bf16) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const size_t per_row = cols >> 3;
  if (i >= (size_t)rows * per_row) return;
  const size_t r = i / per_row;
  const int c = (int)(i % per_row) * 8;
  const int ng = (cols + group - 1) / group;
  const uint32_t w = *(const uint32_t*)(q4 + r * (cols >> 1) + (c >> 1));
  const float s = half_bits_to_f32(scale[r * ng + c / group]);
  float f[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) f[j] = (float)nib_s(w, j) * s;
  if (out_f32) {
    float4* o = (float4*)(out_f32 + r * cols + c);
    o[0] = make_float4(f[0], f[1], f[2], f[3]);
    o[1] = make_float4(f[4], f[5], f[6], f[7]);
  }
  if (out_bf16) {
    uint4 v = make_uint4(pack_bf16x2(f[0], f[1]), pack_bf16x2(f[2], f[3]), pack_bf16x2(f[4], f[5]),
                         pack_bf16x2(f[6], f[7]));
    *(uint4*)(out_bf16 + r * cols + c) = v;
  }
}

// x0[n][:] = mul * E[ids[n]][:] decompressed to fp32; one thread per 8 codes.
// An id outside [0, V) yields a NaN row instead of an out-of-bounds read.
__global__ void k_embed(const uint8_t* q4, const uint16_t* scale, int d, int group, const int32_t* ids,
                        int n, int V, float mul, float* x0) {
  const int per_row = d >> 3;
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (size_t)n * per_row) return;
  const int row = (int)(i / per_row), c = (int)(i % per_row) * 8;
  const int id = ids[row];
  if (id < 0 || id >= V) {
    float4* o = (float4*)(x0 + (size_t)row * d + c);
    o[0] = o[1] = make_float4(NAN, NAN, NAN, NAN);
    return;
  }
  const size_t v = (size_t)id;
  const int ng = (d + group - 1) / group;
  const uint32_t w = *(const uint32_t*)(q4 + v * (d >> 1) + (c >> 1));
  const float s = half_bits_to_f32(scale[v * ng + c / group]);
  float f[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) f[j] = (float)nib_s(w, j) * s * mul;  // mul = 1 is exact
  float4* o = (float4*)(x0 + (size_t)row * d + c);
  o[0] = make_float4(f[0], f[1], f[2], f[3]);
  o[1] = make_float4(f[4], f[5], f[6], f[7]);
}

// ------------------------------------------------------------------ RMSNorm
// One wave per row, float4 accesses (d % 4 == 0). Rows of up to 64 * RC float4s are held in
// registers: every load of the row is issued before the reduction and the row is read once.
constexpr int RC = 16;  // rows up to 4096 values take the register path
constexpr int RCB = 12;  // (backward: two row arrays, up to 3072 values)
__global__ __launch_bounds__(256) void k_rmsnorm_fwd(const float* x, const float* w, int n, int d, float eps,
                                                     f16* y, float* rstd_out) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (row >= n) return;
  const float4* xr = (const float4*)(x + (size_t)row * d);
  const float4* wr = (const float4*)w;
  uint2* yr = (uint2*)(y + (size_t)row * d);
  const int d4 = d >> 2;
  float ss = 0.f;
  if (d4 <= 64 * RC) {
    float4 v[RC];
#pragma unroll
    for (int q = 0; q < RC; ++q) {
      const int c = lane + 64 * q;
      v[q] = c < d4 ? xr[c] : make_float4(0.f, 0.f, 0.f, 0.f);
      ss += v[q].x * v[q].x + v[q].y * v[q].y + v[q].z * v[q].z + v[q].w * v[q].w;
    }
    ss = wave_sum(ss);
    const float rs = 1.0f / sqrtf(ss / (float)d + eps);
    if (rstd_out && lane == 0) rstd_out[row] = rs;
#pragma unroll
    for (int q = 0; q < RC; ++q) {
      const int c = lane + 64 * q;
      if (c >= d4) break;
      const float4 g = wr[c];
      yr[c] = make_uint2(pack_f16x2(v[q].x * rs * g.x, v[q].y * rs * g.y),
                         pack_f16x2(v[q].z * rs * g.z, v[q].w * rs * g.w));
    }
    return;
  }
  for (int c = lane; c < d4; c += 64) {
    const float4 v = xr[c];
    ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
  }
  ss = wave_sum(ss);
  const float rs = 1.0f / sqrtf(ss / (float)d + eps);
  if (rstd_out && lane == 0) rstd_out[row] = rs;
  for (int c = lane; c < d4; c += 64) {
    const float4 v = xr[c], g = wr[c];
    yr[c] = make_uint2(pack_f16x2(v.x * rs * g.x, v.y * rs * g.y), pack_f16x2(v.z * rs * g.z, v.w * rs * g.w));
  }
}

// dx = resid + rstd * (w*dy - xhat * mean(xhat*w*dy)), xhat = x*rstd (weight frozen).
__global__ __launch_bounds__(256) void k_rmsnorm_bwd(const float* x, const float* w, const float* dy,
                                                     const float* resid, int n, int d, float eps, float* dx,
                                                     bf16* dxb) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (row >= n) return;
  const size_t off = (size_t)row * d;
  const float4* xr = (const float4*)(x + off);
  const float4* gr = (const float4*)(dy + off);
  const float4* wr = (const float4*)w;
  const int d4 = d >> 2;
  float ss = 0.f, sd = 0.f;
  const float4* rr = (const float4*)(resid ? resid + off : nullptr);
  float4* o = dx ? (float4*)(dx + off) : nullptr;
  uint2* ob = dxb ? (uint2*)(dxb + off) : nullptr;
  if (d4 <= 64 * RCB) {
    // rows of up to 64 * RCB float4s: x and dy held in registers, every load issued up front
    float4 xv[RCB], gv[RCB];
#pragma unroll
    for (int q = 0; q < RCB; ++q) {
      const int c = lane + 64 * q;
      const bool ok = c < d4;
      xv[q] = ok ? xr[c] : make_float4(0.f, 0.f, 0.f, 0.f);
      gv[q] = ok ? gr[c] : make_float4(0.f, 0.f, 0.f, 0.f);
      const float4 ww = ok ? wr[c] : make_float4(0.f, 0.f, 0.f, 0.f);
      ss += xv[q].x * xv[q].x + xv[q].y * xv[q].y + xv[q].z * xv[q].z + xv[q].w * xv[q].w;
      sd += xv[q].x * ww.x * gv[q].x + xv[q].y * ww.y * gv[q].y + xv[q].z * ww.z * gv[q].z + xv[q].w * ww.w * gv[q].w;
    }
    ss = wave_sum(ss);
    sd = wave_sum(sd);
    const float rs = 1.0f / sqrtf(ss / (float)d + eps);
    const float mean_term = rs * sd / (float)d;
#pragma unroll
    for (int q = 0; q < RCB; ++q) {
      const int c = lane + 64 * q;
      if (c >= d4) break;
      const float4 v = xv[q], g = gv[q], ww = wr[c];
      float4 res = rr ? rr[c] : make_float4(0.f, 0.f, 0.f, 0.f);
      res.x += rs * (ww.x * g.x - v.x * rs * mean_term);
      res.y += rs * (ww.y * g.y - v.y * rs * mean_term);
      res.z += rs * (ww.z * g.z - v.z * rs * mean_term);
      res.w += rs * (ww.w * g.w - v.w * rs * mean_term);
      if (o) o[c] = res;
      if (ob) ob[c] = make_uint2(pack_bf16x2(res.x, res.y), pack_bf16x2(res.z, res.w));
    }
    return;
  }
  for (int c = lane; c < d4; c += 64) {
    const float4 v = xr[c], g = gr[c], ww = wr[c];
    ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
    sd += v.x * ww.x * g.x + v.y * ww.y * g.y + v.z * ww.z * g.z + v.w * ww.w * g.w;
  }
  ss = wave_sum(ss);
  sd = wave_sum(sd);
  const float rs = 1.0f / sqrtf(ss / (float)d + eps);
  const float mean_term = rs * sd / (float)d;  // mean(xhat * w * dy)
  for (int c = lane; c < d4; c += 64) {
    const float4 v = xr[c], g = gr[c], ww = wr[c];
    float4 res = rr ? rr[c] : make_float4(0.f, 0.f, 0.f, 0.f);
    res.x += rs * (ww.x * g.x - v.x * rs * mean_term);
    res.y += rs * (ww.y * g.y - v.y * rs * mean_term);
    res.z += rs * (ww.z * g.z - v.z * rs * mean_term);
    res.w += rs * (ww.w * g.w - v.w * rs * mean_term);
    if (o) o[c] = res;
    if (ob) ob[c] = make_uint2(pack_bf16x2(res.x, res.y), pack_bf16x2(res.z, res.w));
  }
}

__global__ void k_f32_to_bf16(const float* x, bf16* y, size_t n4) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n4) return;
  const float4 v = ((const float4*)x)[i];
  ((uint2*)y)[i] = make_uint2(pack_bf16x2(v.x, v.y), pack_bf16x2(v.z, v.w));
}

// ------------------------------------------------------------------ RoPE
// cs[t][i] = (cos, sin)(t * theta^(-2i/dh)), computed in fp64.
__global__ void k_rope_table(int T, int dh, double theta, float* cs) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  const int half = dh >> 1;
  if (i >= T * half) return;
  const int t = i / half, j = i % half;
  const double inv = pow(theta, -(2.0 * j) / (double)dh);
  const double ang = (double)t * inv;
  cs[2 * i] = (float)cos(ang);
  cs[2 * i + 1] = (float)sin(ang);
}

// z = act(g) * u, 8 elements per thread
__global__ void k_act_fwd(const f16* g, const f16* u, f16* z, size_t n8, int act) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n8) return;
  const uint4 gv = ((const uint4*)g)[i], uv = ((const uint4*)u)[i];
  const uint32_t* gp = (const uint32_t*)&gv;
  const uint32_t* up = (const uint32_t*)&uv;
  uint32_t o[4];
#pragma unroll
  for (int j = 0; j < 4; ++j)
    o[j] = pack_f16x2(act_f(f16_lo(gp[j]), act) * f16_lo(up[j]), act_f(f16_hi(gp[j]), act) * f16_hi(up[j]));
  ((uint4*)z)[i] = make_uint4(o[0], o[1], o[2], o[3]);
}

// ------------------------------------------------------------------ cross-entropy
// tgt[b*T+t] = ids[b][t+1] for t < T-1, -1 (no target) for t = T-1; an id outside
// [0, V) becomes -2, which the loss turns into NaN instead of an out-of-bounds read.
__global__ void k_targets(const int32_t* ids, int B, int T, int V, int32_t* tgt) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= B * T) return;
  const int t = i % T;
  int v = -1;
  if (t < T - 1) {
    v = ids[i + 1];
    if (v < 0 || v >= V) v = -2;
  }
  tgt[i] = v;
}

// The LM head runs over the vocabulary in chunks (columns [v0, v0 + w) at a time) with
// per-row running statistics: m = the largest logit so far, l = sum of exp(logit - m) so
// far. The logits GEMM leaves per (row, 64-column tile) its maximum and its sum of
// exp(logit - max), and the logits themselves relative to that maximum (fp16).

// One wave per row: the chunk's (max, sum) from its tiles, merged into the running (m, l);
// alpha = exp(m_old - m_new), the factor that moves the row's dH accumulator to the new
// maximum (unused on the first chunk, which sets m and l).
__global__ __launch_bounds__(256) void k_ce_chunk_stats(const float2* stats, int ld, int nt, int M, float* mrun,
                                                        float* lrun, float* alpha, int first) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (row >= M) return;
  const float2* st = stats + (size_t)row * ld;
  float mx = -INFINITY;
  for (int i = lane; i < nt; i += 64) mx = fmaxf(mx, st[i].x);
  mx = wave_max(mx);
  float se = 0.f;
  for (int i = lane; i < nt; i += 64) se += st[i].y * __expf(st[i].x - mx);
  se = wave_sum(se);
  if (lane == 0) {
    if (first) {
      mrun[row] = mx;
      lrun[row] = se;
      alpha[row] = 0.f;
    } else {
      const float mo = mrun[row], mn = fmaxf(mo, mx);
      const float a = __expf(mo - mn);
      lrun[row] = lrun[row] * a + se * __expf(mx - mn);
      mrun[row] = mn;
      alpha[row] = a;
    }
  }
}

__global__ __launch_bounds__(256) void k_ce_loss(const float* row_loss, int M, float inv_n, float* loss) {
  __shared__ float red[4];
  float acc = 0.f;
  for (int i = threadIdx.x; i < M; i += 256) acc += row_loss[i];
  acc = wave_sum(acc);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) loss[0] = ((red[0] + red[1]) + (red[2] + red[3])) * inv_n;
}

// Copy between device memory and pinned host memory (its device address) by a few
// workgroups (16-byte accesses, grid-stride): the host link, not the chip, bounds it, so it
// needs few compute units, and unlike a copy kernel sized to the buffer it leaves the others
// to the layer kernels running beside it. 8192 threads keep 128 KB in flight, enough for the
// link's bandwidth-latency product.
constexpr int COPY_WGS = 32;
__global__ __launch_bounds__(256) void k_copy_host(const uint4* __restrict__ src, uint4* __restrict__ dst,
                                                   size_t n16) {
  for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n16; i += (size_t)COPY_WGS * 256) dst[i] = src[i];
}

// Unnormalised softmax weights of one vocabulary chunk, written in place over its fp16
// logits as the bf16 A operand of the dH product: p = exp(logit - m) with m the row's
// running maximum after this chunk (logit - m = stored value + tile maximum - m, so the
// fp16 rounding applies to the small tile-relative value only). The target column is
// left out (0): its term (P_target - 1) E[target] is added in fp32 by k_ce_final, so the
// cancellation of a confident row's gradient does not go through 16-bit operands. Rows
// without a target get zeros. One thread per 8 columns (w % 8 == 0, rows 16-byte aligned).
__global__ __launch_bounds__(256) void k_ce_probs(uint16_t* lg, int M, int w, int ld, const float2* stats,
                                                  int ld_tiles, const float* mrun, const int32_t* tgt, int v0) {
  const int per_row = w >> 3;
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (size_t)M * per_row) return;
  const int m = (int)(i / per_row), c = (int)(i % per_row) * 8;
  uint4* p = reinterpret_cast<uint4*>(lg + (size_t)m * ld + c);
  const int tg = tgt[m];
  uint4 o = make_uint4(0, 0, 0, 0);
  if (tg >= 0) {
    const float shift = stats[(size_t)m * ld_tiles + (c >> 6)].x - mrun[m];
    const uint4 h = *p;
    const uint32_t hw[4] = {h.x, h.y, h.z, h.w};
    float e[8];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      e[2 * j] = __expf(f16_lo(hw[j]) + shift);
      e[2 * j + 1] = __expf(f16_hi(hw[j]) + shift);
    }
    const int tl = tg - v0 - c;
    if (tl >= 0 && tl < 8) e[tl] = 0.f;
    o = make_uint4(pack_bf16x2(e[0], e[1]), pack_bf16x2(e[2], e[3]), pack_bf16x2(e[4], e[5]), pack_bf16x2(e[6], e[7]));
  }
  *p = o;
}

// dH accumulator of the LM head: dh = (first ? 0 : alpha[m] dh) + sum_s part[s] (split-K
// planes of this chunk's product, summed in split order). One thread per 4 values.
__global__ __launch_bounds__(256) void k_ce_dh_accum(const float* part, int splits, int M, int d, const float* alpha,
                                                     int first, float* dh) {
  const size_t n4 = (size_t)M * d / 4;
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n4) return;
  float4 v = ((const float4*)part)[i];
  for (int s = 1; s < splits; ++s) {
    const float4 t = ((const float4*)part)[(size_t)s * n4 + i];
    v.x += t.x; v.y += t.y; v.z += t.z; v.w += t.w;
  }
  if (!first) {
    const float a = alpha[(i * 4) / d];
    const float4 o = ((const float4*)dh)[i];
    v.x += a * o.x; v.y += a * o.y; v.z += a * o.z; v.w += a * o.w;
  }
  ((float4*)dh)[i] = v;
}

// End of the LM head, per row: lse = m + log l, the row's loss term lse - logit[target],
// and, in place, dhf = inv_n (dh / l + (P_target - 1) E[target]) with P_target - 1 =
// expm1(logit[target] - lse) and E[target] decompressed exactly in fp32; rows without a
// target get zeros, an id outside [0, V) a NaN loss term. One thread per 8 columns.
__global__ __launch_bounds__(256) void k_ce_final(int M, int d, const uint8_t* eq4, const uint16_t* escale,
                                                  const int32_t* tgt, const float* tgt_logit, const float* mrun,
                                                  const float* lrun, float inv_n, float* dhf, float* lse,
                                                  float* row_loss) {
  const int per_row = d >> 3;
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (size_t)M * per_row) return;
  const int m = (int)(i / per_row), c = (int)(i % per_row) * 8;
  const int tg = tgt[m];
  const float l = lrun[m], L = mrun[m] + logf(l);
  if (c == 0) {
    lse[m] = L;
    row_loss[m] = tg >= 0 ? L - tgt_logit[m] : (tg == -1 ? 0.f : NAN);
  }
  float4* out = (float4*)(dhf + (size_t)m * d + c);
  if (tg < 0) {
    out[0] = out[1] = make_float4(0.f, 0.f, 0.f, 0.f);
    return;
  }
  const float pt1 = expm1f(tgt_logit[m] - L), inv_l = 1.0f / l;
  const int ng = (d + 31) >> 5;
  const uint32_t w = *(const uint32_t*)(eq4 + (size_t)tg * (d >> 1) + (c >> 1));
  const float s = half_bits_to_f32(escale[(size_t)tg * ng + (c >> 5)]);
  const float4 a = out[0], b = out[1];
  const float h[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
  float o[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) o[j] = inv_n * (h[j] * inv_l + pt1 * ((float)nib_s(w, j) * s));
  out[0] = make_float4(o[0], o[1], o[2], o[3]);
  out[1] = make_float4(o[4], o[5], o[6], o[7]);
}

inline unsigned blocks_for(size_t n, unsigned bs) { return (unsigned)((n + bs - 1) / bs); }

// ------------------------------------------------------------------ architecture extras
// out = resid + RMSNorm(t) * w, one wave per row (the sandwich norms of the attention and
// MLP outputs before the residual add).
__global__ __launch_bounds__(256) void k_resid_rmsnorm(const float* resid, const float* t, const float* w, int n,
                                                       int d, float eps, float* out) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (row >= n) return;
  const size_t off = (size_t)row * d;
  const float4* tr = (const float4*)(t + off);
  const int d4 = d >> 2;
  float ss = 0.f;
  for (int c = lane; c < d4; c += 64) {
    const float4 v = tr[c];
    ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
  }
  ss = wave_sum(ss);
  const float rs = 1.0f / sqrtf(ss / (float)d + eps);
  const float4* rr = (const float4*)(resid + off);
  const float4* wr = (const float4*)w;
  float4* o = (float4*)(out + off);
  for (int c = lane; c < d4; c += 64) {
    const float4 v = tr[c], g = wr[c], r = rr[c];
    o[c] = make_float4(r.x + v.x * rs * g.x, r.y + v.y * rs * g.y, r.z + v.z * rs * g.z, r.w + v.w * rs * g.w);
  }
}

// q, k heads after their projections (fp16, in place): + bias, then (with a norm weight)
// RMSNorm over the head keeping the pre-norm values in `pre`, then RoPE; v: + bias. One
// thread per (row, head, 4 columns e of the first half and their partners e + dh/2); the
// dh/8 threads of a head are consecutive lanes and reduce with butterfly shuffles.
__global__ void k_qkv_post(f16* x, int ld, int n, int T, int H, int dh, const float* bias, const float* nw,
                           float eps, f16* pre, const float* cs, int rope) {
  const int G = dh >> 3, half = dh >> 1;
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const bool ok = i < (size_t)n * H * G;
  const int j = (int)(i % G), e = 4 * j;
  const int h = (int)((i / G) % H);
  const size_t row = i / ((size_t)G * H);
  float lo[4] = {0, 0, 0, 0}, hi[4] = {0, 0, 0, 0};
  f16* p = x + row * ld + h * dh;
  if (ok) {
    const uint2 a = *(const uint2*)(p + e), b = *(const uint2*)(p + e + half);
    lo[0] = f16_lo(a.x); lo[1] = f16_hi(a.x); lo[2] = f16_lo(a.y); lo[3] = f16_hi(a.y);
    hi[0] = f16_lo(b.x); hi[1] = f16_hi(b.x); hi[2] = f16_lo(b.y); hi[3] = f16_hi(b.y);
    if (bias) {
      const float4 b1 = *(const float4*)(bias + h * dh + e), b2 = *(const float4*)(bias + h * dh + e + half);
      lo[0] += b1.x; lo[1] += b1.y; lo[2] += b1.z; lo[3] += b1.w;
      hi[0] += b2.x; hi[1] += b2.y; hi[2] += b2.z; hi[3] += b2.w;
    }
  }
  if (nw) {
    if (ok) {
      // the pre-norm values are kept in fp16 and the statistics computed from exactly those
      // values, which the backward reads again
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        lo[t] = (float)(f16)lo[t];
        hi[t] = (float)(f16)hi[t];
      }
      f16* q = pre + row * ld + h * dh;
      *(uint2*)(q + e) = make_uint2(pack_f16x2(lo[0], lo[1]), pack_f16x2(lo[2], lo[3]));
      *(uint2*)(q + e + half) = make_uint2(pack_f16x2(hi[0], hi[1]), pack_f16x2(hi[2], hi[3]));
    }
    float ss = 0.f;
#pragma unroll
    for (int t = 0; t < 4; ++t) ss += lo[t] * lo[t] + hi[t] * hi[t];
    for (int m = 1; m < G; m <<= 1) ss += __shfl_xor(ss, m, 64);
    const float rs = 1.0f / sqrtf(ss / (float)dh + eps);
    if (ok) {
      const float4 w1 = *(const float4*)(nw + e), w2 = *(const float4*)(nw + e + half);
      lo[0] *= rs * w1.x; lo[1] *= rs * w1.y; lo[2] *= rs * w1.z; lo[3] *= rs * w1.w;
      hi[0] *= rs * w2.x; hi[1] *= rs * w2.y; hi[2] *= rs * w2.z; hi[3] *= rs * w2.w;
    }
  }
  if (!ok) return;
  if (rope) {
    const int t = (int)(row % T);
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const float c = cs[2 * (t * half + e + u)], sn = cs[2 * (t * half + e + u) + 1];
      const float x1 = lo[u], x2 = hi[u];
      lo[u] = x1 * c - x2 * sn;
      hi[u] = x2 * c + x1 * sn;
    }
  }
  *(uint2*)(p + e) = make_uint2(pack_f16x2(lo[0], lo[1]), pack_f16x2(lo[2], lo[3]));
  *(uint2*)(p + e + half) = make_uint2(pack_f16x2(hi[0], hi[1]), pack_f16x2(hi[2], hi[3]));
}

// RoPE in place on fp16 q or k (rotate-half pairs (e, e + dh/2), angles from the cos/sin
// table of the row's position). One thread per (row, 8 columns e of the first half): the
// table entries of those columns are read once (four 16-byte loads) and applied to every
// head of the row, 16-byte accesses to the values.
__global__ void k_rope_fwd(f16* x, int ld, int n, int T, int H, int dh, const float* cs) {
  const int half = dh >> 1, C = half >> 3;
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (size_t)n * C) return;
  const int e = 8 * (int)(i % C);
  const size_t row = i / C;
  const int t = (int)(row % T);
  const float4* tp = (const float4*)(cs + 2 * ((size_t)t * half + e));
  float c[8], sn[8];
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const float4 v = tp[u];
    c[2 * u] = v.x; sn[2 * u] = v.y; c[2 * u + 1] = v.z; sn[2 * u + 1] = v.w;
  }
  f16* p = x + row * ld + e;
  for (int h = 0; h < H; ++h, p += dh) {
    const uint4 a = *(const uint4*)p, b = *(const uint4*)(p + half);
    const uint32_t av[4] = {a.x, a.y, a.z, a.w}, bv[4] = {b.x, b.y, b.z, b.w};
    uint32_t lo[4], hi[4];
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const float x1a = f16_lo(av[w]), x1b = f16_hi(av[w]), x2a = f16_lo(bv[w]), x2b = f16_hi(bv[w]);
      const int u0 = 2 * w, u1 = 2 * w + 1;
      lo[w] = pack_f16x2(x1a * c[u0] - x2a * sn[u0], x1b * c[u1] - x2b * sn[u1]);
      hi[w] = pack_f16x2(x2a * c[u0] + x1a * sn[u0], x2b * c[u1] + x1b * sn[u1]);
    }
    *(uint4*)p = make_uint4(lo[0], lo[1], lo[2], lo[3]);
    *(uint4*)(p + half) = make_uint4(hi[0], hi[1], hi[2], hi[3]);
  }
}

// Per-head RMSNorm backward in place on the gradient g (bf16) from the stored pre-norm
// values (fp16): g = rstd * (w*g - xhat * mean(xhat*w*g)). Thread mapping as k_qkv_post.
__global__ void k_headnorm_bwd(const f16* pre, int ld, int n, int H, int dh, const float* nw, float eps, bf16* g,
                               int ldg) {
  const int G = dh >> 3, half = dh >> 1;
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const bool ok = i < (size_t)n * H * G;
  const int j = (int)(i % G), e = 4 * j;
  const int h = (int)((i / G) % H);
  const size_t row = i / ((size_t)G * H);
  float xv[8] = {0, 0, 0, 0, 0, 0, 0, 0}, gv[8] = {0, 0, 0, 0, 0, 0, 0, 0}, wv[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  const f16* xp = pre + row * ld + h * dh;
  bf16* gp = g + row * ldg + h * dh;
  if (ok) {
    const uint2 a = *(const uint2*)(xp + e), b = *(const uint2*)(xp + e + half);
    const uint2 c = *(const uint2*)(gp + e), d = *(const uint2*)(gp + e + half);
    xv[0] = f16_lo(a.x); xv[1] = f16_hi(a.x); xv[2] = f16_lo(a.y); xv[3] = f16_hi(a.y);
    xv[4] = f16_lo(b.x); xv[5] = f16_hi(b.x); xv[6] = f16_lo(b.y); xv[7] = f16_hi(b.y);
    gv[0] = bf16_lo(c.x); gv[1] = bf16_hi(c.x); gv[2] = bf16_lo(c.y); gv[3] = bf16_hi(c.y);
    gv[4] = bf16_lo(d.x); gv[5] = bf16_hi(d.x); gv[6] = bf16_lo(d.y); gv[7] = bf16_hi(d.y);
    const float4 w1 = *(const float4*)(nw + e), w2 = *(const float4*)(nw + e + half);
    wv[0] = w1.x; wv[1] = w1.y; wv[2] = w1.z; wv[3] = w1.w; wv[4] = w2.x; wv[5] = w2.y; wv[6] = w2.z; wv[7] = w2.w;
  }
  float ss = 0.f, sd = 0.f;
#pragma unroll
  for (int t = 0; t < 8; ++t) {
    ss += xv[t] * xv[t];
    sd += xv[t] * wv[t] * gv[t];
  }
  for (int m = 1; m < G; m <<= 1) {
    ss += __shfl_xor(ss, m, 64);
    sd += __shfl_xor(sd, m, 64);
  }
  if (!ok) return;
  const float rs = 1.0f / sqrtf(ss / (float)dh + eps);
  const float mt = rs * sd / (float)dh;  // mean(xhat * w * g)
  float o[8];
#pragma unroll
  for (int t = 0; t < 8; ++t) o[t] = rs * (wv[t] * gv[t] - xv[t] * rs * mt);
  *(uint2*)(gp + e) = make_uint2(pack_bf16x2(o[0], o[1]), pack_bf16x2(o[2], o[3]));
  *(uint2*)(gp + e + half) = make_uint2(pack_bf16x2(o[4], o[5]), pack_bf16x2(o[6], o[7]));
}

}  // namespace

hipError_t launch_dequant(const uint8_t* q4, const uint16_t* scale, int rows, int cols, int group,
                          float* out_f32, uint16_t* out_bf16, hipStream_t st) {
  const size_t n = (size_t)rows * (cols >> 3);
  if (n == 0) return hipSuccess;
  MEBP_TIMED(st, "dequant", 0.0, (double)n * 4 * (1 + (out_f32 ? 32 : 0) + (out_bf16 ? 16 : 0)),
             hipLaunchKernelGGL(k_dequant, dim3(blocks_for(n, 256)), dim3(256), 0, st, q4, scale, rows, cols, group, out_f32,
                     out_bf16));
  return hipGetLastError();
}
hipError_t launch_embed(const uint8_t* q4, const uint16_t* scale, int d, int group, const int32_t* ids, int n,
                        int V, float* x0, hipStream_t st, float mul) {
  const size_t tot = (size_t)n * (d >> 3);
  MEBP_TIMED(st, "embed", 0.0, (double)tot * 36,
             hipLaunchKernelGGL(k_embed, dim3(blocks_for(tot, 256)), dim3(256), 0, st, q4, scale, d, group, ids, n, V, mul,
                                x0));
  return hipGetLastError();
}
hipError_t launch_resid_rmsnorm(const float* resid, const float* t, const float* w, int n, int d, float eps,
                                float* out, hipStream_t st) {
  MEBP_TIMED(st, "resid_rmsnorm", 0.0, (double)n * d * 16,
             hipLaunchKernelGGL(k_resid_rmsnorm, dim3(blocks_for(n, 4)), dim3(256), 0, st, resid, t, w, n, d, eps, out));
  return hipGetLastError();
}
hipError_t launch_qkv_post(f16* x, int ld, int n, int T, int H, int dh, const float* bias, const float* nw, float eps,
                           f16* pre, const float* cs, int rope, hipStream_t st) {
  const size_t tot = (size_t)n * H * (dh >> 3);
  MEBP_TIMED(st, "qkv_post", 0.0, (double)n * H * dh * (nw ? 6 : 4),
             hipLaunchKernelGGL(k_qkv_post, dim3(blocks_for(tot, 256)), dim3(256), 0, st, x, ld, n, T, H, dh, bias, nw, eps,
                                pre, cs, rope));
  return hipGetLastError();
}
hipError_t launch_headnorm_bwd(const f16* pre, int ld, int n, int H, int dh, const float* nw, float eps, bf16* g,
                               int ldg, hipStream_t st) {
  const size_t tot = (size_t)n * H * (dh >> 3);
  MEBP_TIMED(st, "headnorm_bwd", 0.0, (double)n * H * dh * 6,
             hipLaunchKernelGGL(k_headnorm_bwd, dim3(blocks_for(tot, 256)), dim3(256), 0, st, pre, ld, n, H, dh, nw, eps, g,
                                ldg));
  return hipGetLastError();
}
hipError_t launch_rmsnorm_fwd(const float* x, const float* w, int n, int d, float eps, f16* y, float* rstd,
                              hipStream_t st) {
  MEBP_TIMED(st, "rmsnorm_fwd", 0.0, (double)n * d * 6,
             hipLaunchKernelGGL(k_rmsnorm_fwd, dim3(blocks_for(n, 4)), dim3(256), 0, st, x, w, n, d, eps, y, rstd));
  return hipGetLastError();
}
hipError_t launch_rmsnorm_bwd(const float* x, const float* w, const float* dy, const float* resid, int n, int d,
                              float eps, float* dx, bf16* dxb, hipStream_t st) {
  MEBP_TIMED(st, "rmsnorm_bwd", 0.0, (double)n * d * ((resid ? 16 : 12) + (dxb ? 2 : 0)),
             hipLaunchKernelGGL(k_rmsnorm_bwd, dim3(blocks_for(n, 4)), dim3(256), 0, st, x, w, dy, resid, n, d, eps, dx, dxb));
  return hipGetLastError();
}
hipError_t launch_f32_to_bf16(const float* x, bf16* y, size_t n, hipStream_t st) {
  const size_t n4 = n >> 2;
  MEBP_TIMED(st, "f32_to_bf16", 0.0, (double)n4 * 24,
             hipLaunchKernelGGL(k_f32_to_bf16, dim3(blocks_for(n4, 256)), dim3(256), 0, st, x, y, n4));
  return hipGetLastError();
}
hipError_t launch_rope_table(int T, int dh, double theta, float* cs, hipStream_t st) {
  MEBP_TIMED(st, "rope_table", 0.0, (double)T * dh * 4,
             hipLaunchKernelGGL(k_rope_table, dim3(blocks_for((size_t)T * (dh / 2), 256)), dim3(256), 0, st, T, dh, theta, cs));
  return hipGetLastError();
}
hipError_t launch_rope_fwd(f16* x, int ld, int B, int T, int H, int dh, const float* cs, hipStream_t st) {
  const int n = B * T;
  if ((ld & 7) || (dh & 15) || ((uintptr_t)x & 15)) return hipErrorInvalidValue;  // 16-byte accesses
  const size_t tot = (size_t)n * (dh >> 4);
  MEBP_TIMED(st, "rope_fwd", 0.0, (double)n * H * dh * 4,
             hipLaunchKernelGGL(k_rope_fwd, dim3(blocks_for(tot, 256)), dim3(256), 0, st, x, ld, n, T, H, dh, cs));
  return hipGetLastError();
}
hipError_t launch_act_fwd(const f16* g, const f16* u, f16* z, size_t n, int act, hipStream_t st) {
  const size_t n8 = n >> 3;
  MEBP_TIMED(st, "act_fwd", 0.0, (double)n8 * 48,
             hipLaunchKernelGGL(k_act_fwd, dim3(blocks_for(n8, 256)), dim3(256), 0, st, g, u, z, n8, act));
  return hipGetLastError();
}
hipError_t launch_targets(const int32_t* ids, int B, int T, int V, int32_t* tgt, hipStream_t st) {
  MEBP_TIMED(st, "targets", 0.0, (double)B * T * 8,
             hipLaunchKernelGGL(k_targets, dim3(blocks_for((size_t)B * T, 256)), dim3(256), 0, st, ids, B, T, V, tgt));
  return hipGetLastError();
}
hipError_t launch_ce_chunk_stats(const float2* stats, int ld, int nt, int M, float* mrun, float* lrun, float* alpha,
                                 int first, hipStream_t st) {
  MEBP_TIMED(st, "ce_chunk_stats", 0.0, (double)M * nt * 8 + (double)M * 12,
             hipLaunchKernelGGL(k_ce_chunk_stats, dim3(blocks_for(M, 4)), dim3(256), 0, st, stats, ld, nt, M, mrun, lrun,
                                alpha, first));
  return hipGetLastError();
}
hipError_t launch_ce_loss(const float* row_loss, const int32_t* tgt, int M, float inv_n, float* loss,
                          hipStream_t st) {
  (void)tgt;
  MEBP_TIMED(st, "ce_loss", 0.0, (double)M * 4,
             hipLaunchKernelGGL(k_ce_loss, dim3(1), dim3(256), 0, st, row_loss, M, inv_n, loss));
  return hipGetLastError();
}
hipError_t launch_copy_host(const void* src, void* dst, size_t bytes, hipStream_t st) {
  if ((bytes & 15) || ((uintptr_t)src & 15) || ((uintptr_t)dst & 15)) return hipErrorInvalidValue;
  MEBP_TIMED(st, "copy_host", 0.0, (double)bytes * 2,
             hipLaunchKernelGGL(k_copy_host, dim3(COPY_WGS), dim3(256), 0, st, (const uint4*)src, (uint4*)dst,
                                bytes >> 4));
  return hipGetLastError();
}
hipError_t launch_ce_probs(uint16_t* logits, int M, int w, int ld, const float2* stats, int ld_tiles,
                           const float* mrun, const int32_t* tgt, int v0, hipStream_t st) {
  if ((w & 7) || (ld & 7)) return hipErrorInvalidValue;
  const size_t tot = (size_t)M * (w >> 3);
  MEBP_TIMED(st, "ce_probs", 0.0, (double)M * w * 4,
             hipLaunchKernelGGL(k_ce_probs, dim3(blocks_for(tot, 256)), dim3(256), 0, st, logits, M, w, ld, stats,
                                ld_tiles, mrun, tgt, v0));
  return hipGetLastError();
}
hipError_t launch_ce_dh_accum(const float* part, int splits, int M, int d, const float* alpha, int first, float* dh,
                              hipStream_t st) {
  if (d & 3) return hipErrorInvalidValue;
  const size_t n4 = (size_t)M * d / 4;
  MEBP_TIMED(st, "ce_dh_accum", 0.0, (double)n4 * 16 * (splits + (first ? 1 : 2)),
             hipLaunchKernelGGL(k_ce_dh_accum, dim3(blocks_for(n4, 256)), dim3(256), 0, st, part, splits, M, d, alpha,
                                first, dh));
  return hipGetLastError();
}
hipError_t launch_ce_final(int M, int d, const uint8_t* eq4, const uint16_t* escale, const int32_t* tgt,
                           const float* tgt_logit, const float* mrun, const float* lrun, float inv_n, float* dhf,
                           float* lse, float* row_loss, hipStream_t st) {
  if (d & 7) return hipErrorInvalidValue;
  const size_t tot = (size_t)M * (d >> 3);
  MEBP_TIMED(st, "ce_final", 0.0, (double)M * d * 8.5,
             hipLaunchKernelGGL(k_ce_final, dim3(blocks_for(tot, 256)), dim3(256), 0, st, M, d, eq4, escale, tgt,
                                tgt_logit, mrun, lrun, inv_n, dhf, lse, row_loss));
  return hipGetLastError();
}
}  // namespace mebp
