// Device-side helpers shared by the gfx950 kernels of libmebp.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16;
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));

#define DEV static __device__ __forceinline__

DEV int lane_id() { return threadIdx.x & 63; }

// fp32 -> bf16, round to nearest even (v_cvt_pk_bf16_f32 on gfx950).
DEV bf16 to_bf16(float x) { return (bf16)x; }
DEV float bf2f(bf16 x) { return (float)x; }
DEV uint32_t pack_bf16x2(float lo, float hi) {
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  bf16x2 p = {(bf16)lo, (bf16)hi};
  return __builtin_bit_cast(uint32_t, p);
}
DEV float bf16_lo(uint32_t w) { return __builtin_bit_cast(float, w << 16); }
DEV float bf16_hi(uint32_t w) { return __builtin_bit_cast(float, w & 0xffff0000u); }
DEV float half_bits_to_f32(uint16_t h) { return (float)__builtin_bit_cast(_Float16, h); }
// fp32 -> fp16, round to nearest even.
DEV uint32_t pack_f16x2(float lo, float hi) {
  typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
  f16x2 p = {(_Float16)lo, (_Float16)hi};
  return __builtin_bit_cast(uint32_t, p);
}
DEV float f16_lo(uint32_t w) { return (float)__builtin_bit_cast(_Float16, (uint16_t)(w & 0xffffu)); }
DEV float f16_hi(uint32_t w) { return (float)__builtin_bit_cast(_Float16, (uint16_t)(w >> 16)); }
// two fp16 -> two bf16 (round to nearest even)
DEV uint32_t f16x2_to_bf16x2(uint32_t w) { return pack_bf16x2(f16_lo(w), f16_hi(w)); }
DEV uint4 f16x8_to_bf16x8(uint4 v) {
  return make_uint4(f16x2_to_bf16x2(v.x), f16x2_to_bf16x2(v.y), f16x2_to_bf16x2(v.z), f16x2_to_bf16x2(v.w));
}

// Operand element types of the two MFMA flavours used here.
struct OpF16 {
  static __device__ __forceinline__ uint32_t pack(float lo, float hi) { return pack_f16x2(lo, hi); }
  static __device__ __forceinline__ float lo(uint32_t w) { return f16_lo(w); }
  static __device__ __forceinline__ float hi(uint32_t w) { return f16_hi(w); }
};
struct OpBF16 {
  static __device__ __forceinline__ uint32_t pack(float lo, float hi) { return pack_bf16x2(lo, hi); }
  static __device__ __forceinline__ float lo(uint32_t w) { return bf16_lo(w); }
  static __device__ __forceinline__ float hi(uint32_t w) { return bf16_hi(w); }
};

// One 16x16x32 bf16 MFMA: D = A(16x32) * B(32x16) + C.
// Lane l supplies A[l%16][8*(l/16) .. +8] and B[8*(l/16) .. +8][l%16];
// lane l receives D[4*(l/16) + r][l%16], r = 0..3.
DEV f32x4 mfma16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
DEV f32x4 mfma16(f16x8 a, f16x8 b, f32x4 c) { return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0); }
// MFMA on raw 16-byte operands interpreted as Op's element type.
template <class Op>
__device__ __forceinline__ f32x4 mfma16_raw(uint4 a, uint4 b, f32x4 c) {
  if constexpr (__is_same(Op, OpF16))
    return mfma16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), c);
  else
    return mfma16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c);
}

// Signed 4-bit code j (bits [4j, 4j+4)) of a packed dword (v_bfe_i32).
DEV int nib_s(uint32_t w, int j) { return (int)(w << (28 - 4 * j)) >> 28; }

// Decompress 8 int4 codes (one dword, element i in bits [4i, 4i+4)) times scale s into
// 8 16-bit operands (4 dwords, element 2j in the low half of dword j). The product q*s is
// exact in fp32; the conversion to fp16 / bf16 rounds to nearest even.
template <class Op>
DEV uint4 dequant8(uint32_t w, float s) {
  float f[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) f[i] = (float)nib_s(w, i) * s;
  uint4 r;
  r.x = Op::pack(f[0], f[1]);
  r.y = Op::pack(f[2], f[3]);
  r.z = Op::pack(f[4], f[5]);
  r.w = Op::pack(f[6], f[7]);
  return r;
}

DEV float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
DEV float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// Workgroup placement. The dispatcher deals consecutive workgroup ids round-robin to the
// 8 XCDs, each with its own L2. xcd_tile() remaps the ids so that every XCD receives a
// contiguous range of logical tiles (numbered x fastest, then y, then z): tiles that read
// the same row block of the large operand then share one L2 instead of fetching it once per
// XCD. A bijection for any grid size. Used by the large-tile transposed GEMM, whose gradient
// row blocks (up to 20480 wide) are the large operand; the forward GEMMs and the 128x128
// kernels for few tokens keep the plain order, which measured faster there (each XCD then
// touches few weight column blocks; at few tokens everything stays in the last-level cache).
struct TileId {
  int x, y, z;
};
DEV TileId xcd_tile() {
  const int gx = gridDim.x, gy = gridDim.y, total = gx * gy * (int)gridDim.z;
  const int lin = (int)blockIdx.x + gx * ((int)blockIdx.y + gy * (int)blockIdx.z);
  const int xcd = lin & 7, local = lin >> 3, per = total >> 3, rem = total & 7;
  const int logical = xcd < rem ? xcd * (per + 1) + local : rem * (per + 1) + (xcd - rem) * per + local;
  return TileId{logical % gx, (logical / gx) % gy, logical / (gx * gy)};
}

// Raw buffer resources: loads through them return 0 past `bytes` (no per-element bounds
// branches), and offsets are 32-bit VGPR values. Every resource is based at the first row
// a workgroup touches, so a region stays far below 4 GiB.
typedef __amdgpu_buffer_rsrc_t rsrc_t;
DEV rsrc_t make_rsrc(const void* base, size_t bytes) {
  const uint32_t n = bytes > 0xffffffffull ? 0xffffffffu : (uint32_t)bytes;
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)n, 0x00020000);
}
DEV uint4 bload128(rsrc_t r, uint32_t off) {
  typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
  const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, 0);
  return make_uint4(v.x, v.y, v.z, v.w);
}
// with a wave-uniform byte offset added by the buffer unit (no per-lane address arithmetic)
DEV uint4 bload128s(rsrc_t r, uint32_t voff, uint32_t soff) {
  typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
  const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, (int)voff, (int)soff, 0);
  return make_uint4(v.x, v.y, v.z, v.w);
}
DEV uint2 bload64(rsrc_t r, uint32_t off) {
  typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
  const u32x2 v = __builtin_amdgcn_raw_buffer_load_b64(r, (int)off, 0, 0);
  return make_uint2(v.x, v.y);
}
DEV uint32_t bload32(rsrc_t r, uint32_t off) { return __builtin_amdgcn_raw_buffer_load_b32(r, (int)off, 0, 0); }
DEV uint32_t bload16(rsrc_t r, uint32_t off) { return __builtin_amdgcn_raw_buffer_load_b16(r, (int)off, 0, 0); }

// 16-bit element transpose helpers: select the low (or high) halves of two dwords.
DEV uint32_t perm_lo16(uint32_t a, uint32_t b) {  // (a.lo, b.lo) -> lo=a.lo, hi=b.lo
  return __builtin_amdgcn_perm(b, a, 0x05040100u);
}
DEV uint32_t perm_hi16(uint32_t a, uint32_t b) {  // (a.hi, b.hi) -> lo=a.hi, hi=b.hi
  return __builtin_amdgcn_perm(b, a, 0x07060302u);
}

// 2^x by the hardware instruction alone (v_exp_f32; exp2f adds a range check and rescale
// that keep results below 2^-126 as denormals). For softmax weights, which are at most 2^8
// here: results below 2^-126 become 0, which no fp32 sum of them can notice.
DEV float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }

// tanh(x) = 1 - 2 / (exp(2x) + 1) with the hardware exp and reciprocal (absolute error
// around 1e-7, saturating to +-1 for large |x|)
DEV float tanh_fast(float x) { return 1.0f - 2.0f * __builtin_amdgcn_rcpf(__expf(2.0f * x) + 1.0f); }
DEV float sigmoid_fast(float x) { return __builtin_amdgcn_rcpf(1.0f + __expf(-x)); }
DEV float silu_f(float g) { return g * sigmoid_fast(g); }
DEV float gelu_tanh_f(float g) {
  const float c = 0.7978845608028654f;
  return 0.5f * g * (1.0f + tanh_fast(c * (g + 0.044715f * g * g * g)));
}
DEV float act_f(float g, int kind) { return kind == 0 ? silu_f(g) : gelu_tanh_f(g); }
// the same with the kind known at compile time (no branch per element)
template <int KIND>
DEV float act_k(float g) {
  if constexpr (KIND == 0)
    return silu_f(g);
  else
    return gelu_tanh_f(g);
}
DEV float act_grad_f(float g, int kind) {
  if (kind == 0) {
    const float s = sigmoid_fast(g);
    return s * (1.0f + g * (1.0f - s));
  }
  const float c = 0.7978845608028654f;
  const float t = tanh_fast(c * (g + 0.044715f * g * g * g));
  return 0.5f * (1.0f + t) + 0.5f * g * (1.0f - t * t) * c * (1.0f + 3.0f * 0.044715f * g * g);
}
// act(g) and act'(g) of one kind, known at compile time, from one exponential and one
// reciprocal (the same expressions as act_f and act_grad_f)
template <int KIND>
DEV void act_and_grad(float g, float& act, float& grad) {
  if constexpr (KIND == 0) {
    const float s = sigmoid_fast(g);
    act = g * s;
    grad = s * (1.0f + g * (1.0f - s));
  } else {
    const float c = 0.7978845608028654f;
    const float t = tanh_fast(c * (g + 0.044715f * g * g * g));
    act = 0.5f * g * (1.0f + t);
    grad = 0.5f * (1.0f + t) + 0.5f * g * (1.0f - t * t) * c * (1.0f + 3.0f * 0.044715f * g * g);
  }
}
