// Optimizer step on the LoRA parameters: AdamW (decoupled weight decay) and gradient
// accumulation over micro-batches, each over all adapted tensors of all layers in a few
// launches. Both are elementwise streams over fp32 tensors (HBM-bound: AdamW moves 28
// bytes per parameter, accumulation 8 or 12): 16-byte accesses, OPT_VEC float4s per thread
// (a workgroup covers OPT_VEC * 256 consecutive float4s), all loads issued before use. One
// float4 per thread measured fastest: more workgroups per launch hide the ramp-up better
// than more bytes in flight per thread.
//
// The tensors of one launch are listed in a segment table passed as the kernel argument;
// blockIdx.x walks the segments' float4 ranges back to back, and each workgroup finds its
// segment by a scan of the table's block offsets (a workgroup-uniform index).
#include "device_common.h"
#include "mebp_internal.h"

namespace mebp {
namespace {

constexpr int OPT_THREADS = 256, OPT_VEC = 1, OPT_BLOCK = OPT_THREADS * OPT_VEC;

DEV int opt_segment(const OptArgs& a, uint32_t bx) {
  int s = 0;
  while (s + 1 < a.nseg && a.blk0[s + 1] <= bx) ++s;
  return __builtin_amdgcn_readfirstlane(s);
}

DEV float adamw_elem(float p, float g, float& m, float& v, const OptArgs& a) {
  g *= a.grad_scale;
  m = a.beta1 * m + (1.0f - a.beta1) * g;
  v = a.beta2 * v + (1.0f - a.beta2) * g * g;
  const float mh = m * a.inv_bc1, vh = v * a.inv_bc2;
  return p - a.lr * (a.weight_decay * p + mh / (sqrtf(vh) + a.eps));
}

__global__ __launch_bounds__(OPT_THREADS) void k_lora_adamw(const OptArgs a) {
  const int s = opt_segment(a, blockIdx.x);
  const OptSeg& sg = a.seg[s];
  const uint32_t i0 = (blockIdx.x - a.blk0[s]) * OPT_BLOCK + threadIdx.x;
  float4 p[OPT_VEC], m[OPT_VEC], v[OPT_VEC], g[OPT_VEC];
#pragma unroll
  for (int j = 0; j < OPT_VEC; ++j) {
    const uint32_t i = i0 + j * OPT_THREADS;
    if (i < sg.n4) {
      p[j] = ((const float4*)sg.p)[i];
      m[j] = ((const float4*)sg.m)[i];
      v[j] = ((const float4*)sg.v)[i];
      g[j] = ((const float4*)sg.g)[i];
    }
  }
#pragma unroll
  for (int j = 0; j < OPT_VEC; ++j) {
    const uint32_t i = i0 + j * OPT_THREADS;
    if (i >= sg.n4) continue;
    p[j].x = adamw_elem(p[j].x, g[j].x, m[j].x, v[j].x, a);
    p[j].y = adamw_elem(p[j].y, g[j].y, m[j].y, v[j].y, a);
    p[j].z = adamw_elem(p[j].z, g[j].z, m[j].z, v[j].z, a);
    p[j].w = adamw_elem(p[j].w, g[j].w, m[j].w, v[j].w, a);
    ((float4*)sg.p)[i] = p[j];
    ((float4*)sg.m)[i] = m[j];
    ((float4*)sg.v)[i] = v[j];
  }
}

// acc = (first ? 0 : acc) + scale * g   (acc in seg.p, g in seg.g)
__global__ __launch_bounds__(OPT_THREADS) void k_lora_accumulate(const OptArgs a, float scale, int first) {
  const int s = opt_segment(a, blockIdx.x);
  const OptSeg& sg = a.seg[s];
  const uint32_t i0 = (blockIdx.x - a.blk0[s]) * OPT_BLOCK + threadIdx.x;
  float4 g[OPT_VEC], c[OPT_VEC];
#pragma unroll
  for (int j = 0; j < OPT_VEC; ++j) {
    const uint32_t i = i0 + j * OPT_THREADS;
    if (i < sg.n4) {
      g[j] = ((const float4*)sg.g)[i];
      c[j] = first ? make_float4(0.f, 0.f, 0.f, 0.f) : ((const float4*)sg.p)[i];
    }
  }
#pragma unroll
  for (int j = 0; j < OPT_VEC; ++j) {
    const uint32_t i = i0 + j * OPT_THREADS;
    if (i >= sg.n4) continue;
    ((float4*)sg.p)[i] = make_float4(c[j].x + scale * g[j].x, c[j].y + scale * g[j].y, c[j].z + scale * g[j].z,
                                     c[j].w + scale * g[j].w);
  }
}

}  // namespace

// Launches over `segs` in tables of at most OPT_MAXSEG segments (`a` carries the scalar
// parameters; its table fields are filled here).
hipError_t launch_lora_opt(const OptSeg* segs, int nseg, OptArgs a, int mode, float scale, int first,
                           hipStream_t st) {
  double bytes_per_float = mode == 0 ? 28.0 : (first ? 8.0 : 12.0);
  for (int s0 = 0; s0 < nseg; s0 += OPT_MAXSEG) {
    const int n = nseg - s0 < OPT_MAXSEG ? nseg - s0 : OPT_MAXSEG;
    uint32_t blocks = 0;
    double floats = 0;
    for (int j = 0; j < n; ++j) {
      a.seg[j] = segs[s0 + j];
      a.blk0[j] = blocks;
      blocks += (a.seg[j].n4 + OPT_BLOCK - 1) / OPT_BLOCK;
      floats += 4.0 * a.seg[j].n4;
    }
    a.nseg = n;
    if (!blocks) continue;
    if (mode == 0) {
      MEBP_TIMED(st, "lora_adamw", 0.0, floats * bytes_per_float,
                 hipLaunchKernelGGL(k_lora_adamw, dim3(blocks), dim3(OPT_THREADS), 0, st, a));
    } else {
      MEBP_TIMED(st, "lora_grad_accumulate", 0.0, floats * bytes_per_float,
                 hipLaunchKernelGGL(k_lora_accumulate, dim3(blocks), dim3(OPT_THREADS), 0, st, a, scale, first));
    }
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace mebp
