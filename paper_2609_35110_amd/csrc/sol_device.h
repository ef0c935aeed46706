// Device helpers shared by the HIP kernels (sol_kernels.hip, sol_sparse.hip,
// sol_records.hip): token positions on the latent grid, bf16/fp16
// conversions, the 3D rotary embedding of one 16-byte chunk, the QK
// normalisation, the prepared-path tile size and the block-INT8 record
// decoding.  Every rotation and normalisation in the library goes through
// these functions, so all kernels produce the same bits for the same row.
#pragma once

#include "sol_internal.h"

namespace sol {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

constexpr int D = kHeadDim;
constexpr int kChunks = D / 8;  // 16-byte chunks (8 bf16 = 4 rotary pairs) per row

// ------------------------------------------------------------ rotary helpers

// Workgroups are dispatched round-robin over the 8 XCDs (workgroup w runs on
// XCD w % 8), and each XCD has its own L2.  Renumber them so that XCD x gets
// one contiguous range of work items: the workgroups an XCD runs at the same
// time then stream the same (b, h) slab's K and V through its L2 together.
// A bijection on [0, n) for any n.
constexpr int kXcds = 8;
__device__ __forceinline__ int xcd_local_id(int w, int n) {
  const int xcd = w % kXcds, local = w / kXcds;
  const int per = n / kXcds, rem = n % kXcds;
  return xcd < rem ? xcd * (per + 1) + local : rem * (per + 1) + (xcd - rem) * per + local;
}

// n / d for 0 <= n < 2^23, d >= 1: float reciprocal estimate (off by at most
// one) and one integer correction.
__device__ __forceinline__ int div_exact(int n, int d, float inv) {
  int q = (int)((float)n * inv);
  int r = n - q * d;
  q += (r >= d) - (r < 0);
  return q;
}

struct Pos {
  int t, h, w;
  bool rot;  // false for prefix tokens, which are not rotated
};

__device__ __forceinline__ Pos token_pos(int n, const SeqGrid& g) {
  Pos p;
  int r = n - g.nt;
  p.rot = r >= 0;
  r = r < 0 ? 0 : r;
  p.t = div_exact(r, g.hw, g.inv_hw);
  const int rem = r - p.t * g.hw;
  p.h = div_exact(rem, g.Wl, g.inv_wl);
  p.w = rem - p.h * g.Wl;
  return p;
}

// First table pair of 16-byte chunk cc (head dims [8cc, 8cc+8)) at position p,
// under the grid's rotary split (32/48/48 by default: chunks 0-3 carry t, 4-9
// h, 10-15 w).  A chunk past the split passes through: it turns by the pairs
// of a position-0 row, angle 0, (cos, sin) = (1, 0), an exact identity (as
// prefix tokens do, at position (0, 0, 0)).
__device__ __forceinline__ int tab_pair(int cc, const Pos& p, const SeqGrid& g) {
  if (cc < g.c_t) return p.t * g.s_t + 4 * cc;
  if (cc < g.c_h) return g.tab_h + p.h * g.s_h + 4 * (cc - g.c_t);
  if (cc < g.c_w) return g.tab_w + p.w * g.s_w + 4 * (cc - g.c_h);
  return g.id_pair;
}

__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  bf16x2 r;
  r[0] = (__bf16)a;  // v_cvt_pk_bf16_f32: round to nearest even
  r[1] = (__bf16)b;
  return __builtin_bit_cast(uint32_t, r);
}

// bf16 pair (one 32-bit word) -> fp16 pair: exact for |x| < 65504 (fp16
// subnormals below 2^-14 keep 2^-24 absolute resolution).
__device__ __forceinline__ uint32_t bf16x2_to_f16x2(uint32_t w) {
  f16x2 r;
  r[0] = (_Float16)__uint_as_float(w << 16);
  r[1] = (_Float16)__uint_as_float(w & 0xffff0000u);
  return __builtin_bit_cast(uint32_t, r);
}

__device__ __forceinline__ uint4 bf16x8_to_f16x8(uint4 x) {
  return make_uint4(bf16x2_to_f16x2(x.x), bf16x2_to_f16x2(x.y), bf16x2_to_f16x2(x.z),
                    bf16x2_to_f16x2(x.w));
}

// The eight bf16 values of a 16-byte chunk as fp32 (exact), and back (RNE).
__device__ __forceinline__ void unpack_bf16x8(uint4 x, float (&f)[8]) {
  const uint32_t w[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    f[2 * u] = __uint_as_float(w[u] << 16);
    f[2 * u + 1] = __uint_as_float(w[u] & 0xffff0000u);
  }
}
__device__ __forceinline__ uint4 pack_bf16x8(const float (&f)[8]) {
  return make_uint4(pack_bf16x2(f[0], f[1]), pack_bf16x2(f[2], f[3]), pack_bf16x2(f[4], f[5]),
                    pack_bf16x2(f[6], f[7]));
}

// The rotary table (the 3D rotary embedding of Sec. 3.5) is two planes of
// (cos, sin) pairs: plane 0 holds each value rounded to fp32 (hi), plane 1, g.tab_pairs
// pairs on, what that rounding lost (lo = fp32(cos - hi)), so hi + lo carries each
// to 48 bits.
__device__ __forceinline__ const float2* tab_lo_plane(const float2* tab, const SeqGrid& g) {
  return tab ? tab + g.tab_pairs : nullptr;
}

// fp64 -> fp32 rounded to odd: the truncation, its last bit set when inexact.
// With 24 bits against bf16's 8, rounding that to bf16 (nearest even) gives
// the nearest-even bf16 of the double itself: no double-rounding error.
__device__ __forceinline__ float f32_round_odd(double d) {
  const float f = (float)d;  // v_cvt_f32_f64, nearest even
  uint32_t u = __float_as_uint(f);
  const double back = (double)f;
  // inexact and even: the neighbour on d's side (sign-magnitude: +1 is away from 0)
  if (back != d && (u & 1u) == 0) u += fabs(back) < fabs(d) ? 1u : 0xffffffffu;
  return __uint_as_float(u);
}

// Rotate the 4 interleaved pairs of one 16-byte chunk, held as fp32:
//   (a, b) -> (a cos - b sin, a sin + b cos)
// in fp64 with cos and sin taken as hi + lo (48 bits), then one rounding to
// bf16.  The result is the nearest-even bf16 of the exact rotation unless that
// lies within about 2^-47 |(a, b)| of a rounding midpoint.  Every rotation of
// a query or key row in this library goes through this function, except the
// fused kernel's key tiles (rope_rotate_fast below).
__device__ __forceinline__ uint4 rope_rotate_exact(const float (&f)[8], const float2* __restrict__ hi,
                                                   const float2* __restrict__ lo, int pair0) {
  const float4 h01 = *reinterpret_cast<const float4*>(hi + pair0);
  const float4 h23 = *reinterpret_cast<const float4*>(hi + pair0 + 2);
  const float4 l01 = *reinterpret_cast<const float4*>(lo + pair0);
  const float4 l23 = *reinterpret_cast<const float4*>(lo + pair0 + 2);
  // hi + lo is exact in fp64 (|lo| <= half an fp32 ulp of hi)
  const double c[4] = {(double)h01.x + (double)l01.x, (double)h01.z + (double)l01.z,
                       (double)h23.x + (double)l23.x, (double)h23.z + (double)l23.z};
  const double s[4] = {(double)h01.y + (double)l01.y, (double)h01.w + (double)l01.w,
                       (double)h23.y + (double)l23.y, (double)h23.w + (double)l23.w};
  uint32_t w[4];
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const double a = f[2 * u], b = f[2 * u + 1];
    const double ar = __builtin_fma(a, c[u], -(b * s[u]));
    const double br = __builtin_fma(a, s[u], b * c[u]);
    w[u] = pack_bf16x2(f32_round_odd(ar), f32_round_odd(br));
  }
  return make_uint4(w[0], w[1], w[2], w[3]);
}

__device__ __forceinline__ uint4 rope_chunk(uint4 x, const float2* __restrict__ hi,
                                            const float2* __restrict__ lo, int pair0) {
  float f[8];
  unpack_bf16x8(x, f);
  return rope_rotate_exact(f, hi, lo, pair0);
}

// The fused kernel's key tiles: the same rotation in fp32 with the hi plane
// alone (2 VALU operations an element, against about 10 for the exact form,
// in a loop that rotates every key once per query tile).  Within one bf16 ulp
// of rope_rotate_exact; the two differ where the exact result lies within a
// few 2^-24 |(a, b)| of a rounding midpoint.
__device__ __forceinline__ uint4 rope_rotate_fast(uint4 x, float4 cs01, float4 cs23) {
  float f[8];
  unpack_bf16x8(x, f);
  const float c[4] = {cs01.x, cs01.z, cs23.x, cs23.z};
  const float s[4] = {cs01.y, cs01.w, cs23.y, cs23.w};
  uint32_t w[4];
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const float a = f[2 * u], b = f[2 * u + 1];
    const float ar = __builtin_fmaf(a, c[u], -(b * s[u]));
    const float br = __builtin_fmaf(a, s[u], b * c[u]);
    w[u] = pack_bf16x2(ar, br);
  }
  return make_uint4(w[0], w[1], w[2], w[3]);
}

// ------------------------------------------------------- LDS poison (debug)

// Debug build (-DSOL_LDS_POISON): a workgroup first fills the LDS arrays that
// hold values -- never those holding indices, counts or flags -- with NaN bit
// patterns and waits at a barrier, so a read that comes before the write it
// needs (a missing barrier or wait) turns the output to NaN instead of
// quietly reusing stale data.  Compiles to nothing in the normal build.
template <typename T>
__device__ __forceinline__ void lds_poison(T* p, size_t bytes) {
#ifdef SOL_LDS_POISON
  uint32_t* w = reinterpret_cast<uint32_t*>(p);
  for (size_t i = threadIdx.x; i < bytes / 4; i += blockDim.x) w[i] = 0xFFFFFFFFu;
#else
  (void)p;
  (void)bytes;
#endif
}
__device__ __forceinline__ void lds_poison_done() {
#ifdef SOL_LDS_POISON
  __syncthreads();
#endif
}

// ------------------------------------------------------- QK normalization

// RMS normalisation of one head's row ahead of the rotation (Sec. 3.5, fusion
// group 2, "QK normalization with partial RoPE"): x gamma / sqrt(mean(x^2) +
// eps), in fp32, nothing rounded before the rotation.  The sum of squares
// follows one fixed order whichever lanes hold the row -- per 16-byte chunk c
// an fma chain over its eight entries, then a binary tree over the 16 chunk
// sums pairing c with c^1, then c^2, c^4, c^8 -- so every kernel normalises a
// row to the same bits (fp32 addition is commutative, so a butterfly over the
// lanes and a tree inside one lane give the same sums).
__device__ __forceinline__ float chunk_sumsq(uint4 x) {
  float f[8];
  unpack_bf16x8(x, f);
  float s = f[0] * f[0];
#pragma unroll
  for (int e = 1; e < 8; ++e) s = __builtin_fmaf(f[e], f[e], s);
  return s;
}
// The tree over 16 consecutive lanes that hold chunks 0..15 of one row.
__device__ __forceinline__ float row_sumsq_lanes16(float p) {
  p += __shfl_xor(p, 1);
  p += __shfl_xor(p, 2);
  p += __shfl_xor(p, 4);
  p += __shfl_xor(p, 8);
  return p;
}
__device__ __forceinline__ float rms_inv(float sumsq, float eps) {
  return 1.0f / __builtin_sqrtf(sumsq * (1.0f / D) + eps);
}
// Chunk cc (dims 8cc..8cc+7) of a row, normalised: (x inv) gamma, fp32.
__device__ __forceinline__ void norm_chunk(uint4 x, float inv, const float* __restrict__ gamma,
                                           int cc, float (&f)[8]) {
  unpack_bf16x8(x, f);
  const float4 g0 = *reinterpret_cast<const float4*>(gamma + 8 * cc);
  const float4 g1 = *reinterpret_cast<const float4*>(gamma + 8 * cc + 4);
  const float gm[8] = {g0.x, g0.y, g0.z, g0.w, g1.x, g1.y, g1.z, g1.w};
#pragma unroll
  for (int e = 0; e < 8; ++e) f[e] = (f[e] * inv) * gm[e];
}
// Chunk cc of a query or key row as it enters the products: normalised when
// gamma is given (inv from the row's sum of squares), rotated when rot (table
// pairs from pair0 in planes hi and lo), rounded to bf16.
__device__ __forceinline__ uint4 qk_chunk(uint4 x, const float* __restrict__ gamma, float inv, int cc,
                                          bool rot, const float2* __restrict__ hi,
                                          const float2* __restrict__ lo, int pair0) {
  if (gamma == nullptr) return rot ? rope_chunk(x, hi, lo, pair0) : x;
  float f[8];
  norm_chunk(x, inv, gamma, cc, f);
  if (!rot) return pack_bf16x8(f);
  return rope_rotate_exact(f, hi, lo, pair0);
}

// ------------------------------------------------ block-INT8 QKV records

// The wire record of the quantized QKV exchange (Sec. 3.2, "Quantized
// communication"): per (token, head) 400 bytes -- int8 codes of q (bytes
// 0..127), k (128..255) and v (256..383), then one UE5M3 scale code per group
// of 32 values (byte 384 + 4 part + group), then 4 zero bytes.  Records are
// token-major: (b, n, h) at ((b N + n) H + h) 400.  An element is its code
// times its group's scale, rounded once to bf16.
constexpr int kRecBytes = 400;
constexpr int kRecScales = 384;  // first scale byte; part p group g at 384 + 4p + g
// The attention output's block-INT8 record: 128 codes, 4 scale codes (dims
// [32g, 32g + 32)), 12 zero bytes; token-major like the QKV records.
constexpr int kOutRecBytes = 144;

// UE5M3 code -> value: unsigned, 5 exponent bits of bias 15, 3 mantissa bits;
// exponent 0 subnormal (m 2^-17), exponent 31 infinity (m = 0) or NaN.  Exact.
__device__ __forceinline__ float ue5m3_value(uint32_t c) {
  if (c >= 0xF8u) return __uint_as_float(c == 0xF8u ? 0x7F800000u : 0x7FC00000u);
  if (c < 8u) return (float)c * 0x1p-17f;
  return __uint_as_float((c << 20) + (112u << 23));  // exponent e - 15 + 127, mantissa m
}

// Quantisation of a group of 32 values (the records' scale granularity):
// scale s = the smallest finite positive UE5M3 value with 127 s >= max |x|,
// so no code passes +-127; code = x / s rounded to nearest, ties to even.
// 127 s is exact in fp32 (a 4-bit significand times 127), so the scale is
// the exact one, and int8_code rounds the exact quotient x / s, for bf16
// inputs (the QKV records) and fp32 ones (the output epilogue) alike.
// Smallest code c in 1..0xF7 with 127 value(c) >= amax (0xF7 when none is
// large enough).  The candidate is the code at or just above t = amax / 127
// read off t's fp32 bits (exponent and top three mantissa bits, rounded up);
// t's two roundings move it by under 2^-22 of itself while neighbouring codes
// differ by at least 1/16 (2^-17 absolute among the subnormal codes), so the
// candidate is the answer or one code off, and one exact comparison each way
// settles it.
__device__ __forceinline__ uint32_t ue5m3_scale_for(float amax) {
  const float t = amax * (1.0f / 127.0f);
  uint32_t c;
  if (!(t < 61440.0f)) {
    c = 0xF7u;
  } else if (t < 0x1p-14f) {
    c = (uint32_t)__builtin_ceilf(t * 0x1p17f);  // subnormal codes: m 2^-17, m = 0..8
  } else {
    const uint32_t u = __float_as_uint(t);
    c = (u >> 20) - (112u << 3) + ((u & 0xFFFFFu) != 0u);  // (e + 15) << 3 | m, rounded up
  }
  c = c < 1u ? 1u : (c > 0xF7u ? 0xF7u : c);
  if (c > 1u && 127.0f * ue5m3_value(c - 1u) >= amax) --c;
  else if (c < 0xF7u && 127.0f * ue5m3_value(c) < amax) ++c;
  return c;
}
// One value's int8 code at scale s, as the low byte of the result: x / s
// rounded to nearest, ties to even, exactly.  r = rint(x rcp(s)) is the
// answer or one off (the hardware reciprocal's error moves the quotient by
// under 2^-15 here); the residual x - r s is exact (r s lies within a factor
// two of x unless r = 0), so comparing it with s / 2 settles the rounding.
__device__ __forceinline__ uint32_t int8_code(float x, float s) {
  float r = __builtin_rintf(x * __builtin_amdgcn_rcpf(s));
  const float e = __builtin_fmaf(-r, s, x);
  const float h = 0.5f * s, ae = __builtin_fabsf(e);
  if (ae > h || (ae == h && ((int)r & 1) != 0)) r += e > 0.0f ? 1.0f : -1.0f;
  return (uint32_t)(int)fminf(fmaxf(r, -127.0f), 127.0f) & 0xFFu;
}

// Eight int8 codes (one 8-byte word of a record) times their scale, to bf16
// (the product is exact in fp32; one RNE rounding).
__device__ __forceinline__ uint4 decode_rec_chunk(uint2 codes, float s) {
  float f[8];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    f[e] = (float)(int8_t)(codes.x >> (8 * e)) * s;
    f[4 + e] = (float)(int8_t)(codes.y >> (8 * e)) * s;
  }
  return pack_bf16x8(f);
}

// Chunk cc (dims 8cc..8cc+7) of part p (0 q, 1 k, 2 v) of the record at r,
// decoded to bf16.
__device__ __forceinline__ uint4 rec_chunk(const uint8_t* __restrict__ r, int p, int cc) {
  const uint2 codes = *reinterpret_cast<const uint2*>(r + 128 * p + 8 * cc);
  return decode_rec_chunk(codes, ue5m3_value(r[kRecScales + 4 * p + (cc >> 2)]));
}

}  // namespace
}  // namespace sol
