// HIP kernels for gfx950 (CDNA4): standalone 3D rotary embedding and the
// fused rotary + softmax attention forward pass.
//
// Attention layout choices (wave64, v_mfma_f32_32x32x16_bf16):
//   * Scores are computed transposed, S^T = K^ Q^^T, so that in the MFMA
//     result every lane owns ONE query (lane & 31) and 16 of its keys; the
//     other lane half (lane ^ 32) owns the other 16.  Row max and row sum are
//     in-lane plus a single cross-half exchange, and the rescale of the output
//     accumulator is a per-lane scalar.
//   * The output is accumulated transposed too, O^T += V^T P^T: the score
//     registers, rounded to fp16, are directly the B operand (keys along the
//     contraction, in the order the score layout produced them), and the V^T
//     operand is read from a row-major V tile with the gfx950 LDS transpose
//     read (ds_read_b64_tr_b16).
//   * P and V enter the second product as fp16 (V converted exactly from bf16
//     while it is staged): P rounded to bf16 carries a relative error of 2^-9,
//     which on its own nearly doubles the output error of the bf16 result;
//     fp16's 2^-12 leaves the output error at the bf16 output rounding.
//     P <= 2^8 (lazy rescale bound) and |v| < 65504 stay inside fp16's range.
//   * Q^ is rotated once and kept in VGPRs for the whole key sweep; K is
//     rotated while it is staged from HBM into LDS (fused rotary), double
//     buffered, one barrier per 64-key tile.
//   * Online softmax with a lazy rescale: the running max only moves when the
//     new tile max exceeds it by more than 2^8 in probability units, so the
//     64-register output rescale is almost never executed.  Exact: numerator
//     and denominator always share the same reference max.
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

// First table pair of 16-byte chunk cc (head dims [8cc, 8cc+8)) at position p.
// Chunks 0-3 carry t, 4-9 carry h, 10-15 carry w (the 32/48/48 split).
__device__ __forceinline__ int tab_pair(int cc, const Pos& p, const SeqGrid& g) {
  if (cc < 4) return p.t * 16 + 4 * cc;
  if (cc < 10) return g.tab_h + p.h * 24 + 4 * (cc - 4);
  return g.tab_w + p.w * 24 + 4 * (cc - 10);
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

// Rotate the 4 interleaved pairs held in one 16-byte chunk:
//   (a, b) -> (a cos - b sin, a sin + b cos), fp32, then bf16 RNE.
// The one function every rotation in this library goes through, so the
// standalone rotation and the fused tile loads agree bit for bit.
__device__ __forceinline__ uint4 rope_chunk(uint4 x, const float2* __restrict__ tab, int pair0) {
  const float4 cs01 = *reinterpret_cast<const float4*>(tab + pair0);
  const float4 cs23 = *reinterpret_cast<const float4*>(tab + pair0 + 2);
  const float c[4] = {cs01.x, cs01.z, cs23.x, cs23.z};
  const float s[4] = {cs01.y, cs01.w, cs23.y, cs23.w};
  uint32_t w[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const float a = __uint_as_float(w[u] << 16);
    const float b = __uint_as_float(w[u] & 0xffff0000u);
    const float ar = __builtin_fmaf(a, c[u], -(b * s[u]));
    const float br = __builtin_fmaf(a, s[u], b * c[u]);
    w[u] = pack_bf16x2(ar, br);
  }
  return make_uint4(w[0], w[1], w[2], w[3]);
}

// --------------------------------------------------------- standalone rotary

// One thread per 16-byte chunk of one (b, h) slab; grid.y walks the slabs.
__global__ __launch_bounds__(256) void rope3d_kernel(const uint4* __restrict__ x,
                                                     uint4* __restrict__ y, int64_t bh_count,
                                                     SeqGrid g, const float2* __restrict__ tab) {
  const int64_t per_slab = (int64_t)g.n * kChunks;
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= per_slab) return;
  const int n = (int)(i / kChunks);
  const int cc = (int)(i % kChunks);
  const Pos p = token_pos(n, g);
  const int pair0 = p.rot ? tab_pair(cc, p, g) : 0;
  for (int64_t bh = blockIdx.y; bh < bh_count; bh += gridDim.y) {
    const int64_t idx = bh * per_slab + i;
    uint4 v = x[idx];
    if (p.rot) v = rope_chunk(v, tab, pair0);
    y[idx] = v;
  }
}

// ------------------------------------------------------------ fused attention

constexpr int kWaves = 8;
constexpr int kThreads = 64 * kWaves;
constexpr int BM = 32 * kWaves;  // query rows per workgroup (32 per wave)
constexpr int BN = 64;           // keys per tile
constexpr int KS = D + 8;        // K tile row stride in LDS (elements): 272 B
constexpr int VS = D + 16;       // V tile row stride in LDS (elements): 288 B
constexpr float kLazyRescaleLog2 = 8.0f;
static_assert(2 * kThreads == BN * kChunks, "staging: two 16-byte chunks of K and V per thread per tile");

template <bool kRope>
__global__ __launch_bounds__(kThreads, 1) void attn_fwd_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
    const uint16_t* __restrict__ v, uint16_t* __restrict__ out, SeqGrid g,
    const float2* __restrict__ tab, int n_qtiles, float c_log2) {
  __shared__ __attribute__((aligned(16))) uint16_t k_lds[2][BN * KS];
  __shared__ __attribute__((aligned(16))) uint16_t v_lds[2][BN * VS];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int hh = lane >> 5;   // which half of the key block this lane holds
  const int l32 = lane & 31;  // query column of this lane in the score block
  const int bh = blockIdx.x / n_qtiles;
  const int qt = blockIdx.x - bh * n_qtiles;
  const int N = g.n;
  const size_t slab = (size_t)bh * N * D;
  const uint16_t* __restrict__ qs = q + slab;
  const uint16_t* __restrict__ ks = k + slab;
  const uint16_t* __restrict__ vs = v + slab;

  // ---- Q^ fragment (B operand of S^T = K^ Q^^T): dims [16kk + 8hh, +8) of one row.
  const int qrow = qt * BM + wave * 32 + l32;
  bf16x8 qf[8];
  if (qrow < N) {
    const uint4* src = reinterpret_cast<const uint4*>(qs + (size_t)qrow * D);
    Pos p{0, 0, 0, false};
    if (kRope) p = token_pos(qrow, g);
#pragma unroll
    for (int kk = 0; kk < 8; ++kk) {
      const int cc = 2 * kk + hh;
      uint4 x = src[cc];
      if (kRope && p.rot) x = rope_chunk(x, tab, tab_pair(cc, p, g));
      qf[kk] = __builtin_bit_cast(bf16x8, x);
    }
  } else {
#pragma unroll
    for (int kk = 0; kk < 8; ++kk) qf[kk] = __builtin_bit_cast(bf16x8, make_uint4(0, 0, 0, 0));
  }

  // ---- K/V staging: this thread moves chunk column cc_s of tile rows rs0 and rs0 + 32.
  const int cc_s = tid & (kChunks - 1);
  const int rs0 = tid >> 4;
  uint4 kreg[2], vreg[2];
  auto load_tile = [&](int kv0) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int j = kv0 + rs0 + 32 * i;
      if (j < N) {
        kreg[i] = reinterpret_cast<const uint4*>(ks + (size_t)j * D)[cc_s];
        vreg[i] = reinterpret_cast<const uint4*>(vs + (size_t)j * D)[cc_s];
      } else {
        kreg[i] = make_uint4(0, 0, 0, 0);  // keys past N are masked, values must be finite
        vreg[i] = make_uint4(0, 0, 0, 0);
      }
    }
  };
  auto store_tile = [&](int kv0, int buf) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int r = rs0 + 32 * i;
      uint4 kx = kreg[i];
      if (kRope) {
        const int j = kv0 + r;
        if (j < N) {
          const Pos p = token_pos(j, g);
          if (p.rot) kx = rope_chunk(kx, tab, tab_pair(cc_s, p, g));
        }
      }
      *reinterpret_cast<uint4*>(&k_lds[buf][r * KS + cc_s * 8]) = kx;
      *reinterpret_cast<uint4*>(&v_lds[buf][r * VS + cc_s * 8]) = bf16x8_to_f16x8(vreg[i]);
    }
  };

  // V^T operand addressing for the transpose read: within each 16-lane group,
  // lane 4s + c supplies row s (of 4) and 4 columns starting at 4c.
  const int g16 = lane >> 4, i16 = lane & 15;
  const int v_row = 4 * (g16 >> 1) + (i16 >> 2);
  const int v_col = 16 * (g16 & 1) + 4 * (i16 & 3);

  const int n_kv = (N + BN - 1) / BN;
  load_tile(0);
  store_tile(0, 0);
  __syncthreads();

  f32x16 o[4];
#pragma unroll
  for (int db = 0; db < 4; ++db) o[db] = f32x16{};
  float m_run = -__builtin_inff();
  float l_run = 0.0f;

  for (int it = 0; it < n_kv; ++it) {
    const int buf = it & 1;
    const int kv0 = it * BN;
    const bool has_next = it + 1 < n_kv;
    if (has_next) load_tile(kv0 + BN);

    // S^T for key blocks [kv0, kv0+32) and [kv0+32, kv0+64).
    const uint16_t* kb = k_lds[buf];
    f32x16 s0 = f32x16{}, s1 = f32x16{};
#pragma unroll
    for (int kk = 0; kk < 8; ++kk) {
      const bf16x8 a0 = *reinterpret_cast<const bf16x8*>(kb + l32 * KS + kk * 16 + hh * 8);
      const bf16x8 a1 = *reinterpret_cast<const bf16x8*>(kb + (32 + l32) * KS + kk * 16 + hh * 8);
      s0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, qf[kk], s0, 0, 0, 0);
      s1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, qf[kk], s1, 0, 0, 0);
    }
    // Register j of a score block holds key 8(j/4) + 4hh + (j%4) of that block.
    if (kv0 + BN > N) {
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const int key = kv0 + 8 * (j >> 2) + 4 * hh + (j & 3);
        if (key >= N) s0[j] = -__builtin_inff();
        if (key + 32 >= N) s1[j] = -__builtin_inff();
      }
    }

    float mx = fmaxf(s0[0], s1[0]);
#pragma unroll
    for (int j = 1; j < 16; ++j) mx = fmaxf(mx, fmaxf(s0[j], s1[j]));
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float m_new = fmaxf(m_run, mx);
    if (__any((m_new - m_run) * c_log2 > kLazyRescaleLog2)) {
      const float alpha = __builtin_amdgcn_exp2f((m_run - m_new) * c_log2);
      m_run = m_new;
      l_run *= alpha;
#pragma unroll
      for (int db = 0; db < 4; ++db) o[db] *= alpha;
    }
    const float mc = m_run * c_log2;

    // P = exp2(S c - m c), rounded to fp16: the B operand of O^T += V^T P^T.
    f16x8 pb[4];
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(s0[j], c_log2, -mc));
      const float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf(s1[j], c_log2, -mc));
      l_run += p0 + p1;
      pb[j >> 3][j & 7] = (_Float16)p0;
      pb[2 + (j >> 3)][j & 7] = (_Float16)p1;
    }

    // O^T[d, q] += sum over 16-key steps of V^T[d, key] P^T[key, q].
    const uint16_t* vb = v_lds[buf];
#pragma unroll
    for (int kst = 0; kst < 4; ++kst) {
#pragma unroll
      for (int db = 0; db < 4; ++db) {
        const uint16_t* p0 = vb + (16 * kst + v_row) * VS + 32 * db + v_col;
        const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)p0);
        const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p0 + 8 * VS));
        const f16x8 a = __builtin_bit_cast(
            f16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
        o[db] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, pb[kst], o[db], 0, 0, 0);
      }
    }

    if (has_next) store_tile(kv0 + BN, buf ^ 1);
    __syncthreads();
  }

  // ---- epilogue: out = O / l in bf16; register j of block db is dim 32db + 8(j/4) + 4hh + j%4.
  const float l_tot = l_run + __shfl_xor(l_run, 32);
  const float inv = 1.0f / l_tot;
  if (qrow < N) {
    uint16_t* dst = out + slab + (size_t)qrow * D;
#pragma unroll
    for (int db = 0; db < 4; ++db) {
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        uint2 w;
        w.x = pack_bf16x2(o[db][4 * g4] * inv, o[db][4 * g4 + 1] * inv);
        w.y = pack_bf16x2(o[db][4 * g4 + 2] * inv, o[db][4 * g4 + 3] * inv);
        *reinterpret_cast<uint2*>(dst + 32 * db + 8 * g4 + 4 * hh) = w;
      }
    }
  }
}

}  // namespace

hipError_t launch_rope3d(const uint16_t* x, uint16_t* y, int64_t rows, const SeqGrid& g,
                         const float2* tab, hipStream_t stream) {
  const int64_t per_slab = (int64_t)g.n * kChunks;
  const int64_t bh_count = rows / g.n;
  const unsigned gx = (unsigned)((per_slab + 255) / 256);
  const unsigned gy = (unsigned)(bh_count < 65535 ? bh_count : 65535);
  hipLaunchKernelGGL(rope3d_kernel, dim3(gx, gy), dim3(256), 0, stream,
                     reinterpret_cast<const uint4*>(x), reinterpret_cast<uint4*>(y), bh_count, g,
                     tab);
  return hipGetLastError();
}

hipError_t launch_attn_fwd(const uint16_t* q, const uint16_t* k, const uint16_t* v,
                           uint16_t* out, int BH, const SeqGrid& g, const float2* tab,
                           hipStream_t stream) {
  const int n_qtiles = (g.n + BM - 1) / BM;
  const float c_log2 = (float)(1.4426950408889634 / 11.313708498984761);  // log2(e)/sqrt(128)
  const dim3 grid((unsigned)((int64_t)n_qtiles * BH));
  if (tab != nullptr)
    hipLaunchKernelGGL(attn_fwd_kernel<true>, grid, dim3(kThreads), 0, stream, q, k, v, out, g,
                       tab, n_qtiles, c_log2);
  else
    hipLaunchKernelGGL(attn_fwd_kernel<false>, grid, dim3(kThreads), 0, stream, q, k, v, out, g,
                       tab, n_qtiles, c_log2);
  return hipGetLastError();
}

int64_t attn_max_workgroups(int N, int BH) { return (int64_t)((N + BM - 1) / BM) * BH; }

}  // namespace sol
