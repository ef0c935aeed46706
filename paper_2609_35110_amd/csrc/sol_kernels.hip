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
__device__ __forceinline__ uint4 rope_rotate(uint4 x, float4 cs01, float4 cs23) {
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

__device__ __forceinline__ uint4 rope_chunk(uint4 x, const float2* __restrict__ tab, int pair0) {
  return rope_rotate(x, *reinterpret_cast<const float4*>(tab + pair0),
                     *reinterpret_cast<const float4*>(tab + pair0 + 2));
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

// One pass over K and V for the workspace path: K^ = rotated K (bf16, the same
// rounding as the fused tile load), V converted to fp16.  One thread per
// 16-byte chunk of one (b, h) slab; grid.y walks the slabs.
template <bool kRope>
__global__ __launch_bounds__(256) void prep_kv_kernel(const uint4* __restrict__ k,
                                                      const uint4* __restrict__ v,
                                                      uint4* __restrict__ kh, uint4* __restrict__ v16,
                                                      int64_t bh_count, SeqGrid g,
                                                      const float2* __restrict__ tab) {
  const int64_t per_slab = (int64_t)g.n * kChunks;
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= per_slab) return;
  const int n = (int)(i / kChunks);
  const int cc = (int)(i % kChunks);
  const Pos p = kRope ? token_pos(n, g) : Pos{0, 0, 0, false};
  const int pair0 = (kRope && p.rot) ? tab_pair(cc, p, g) : 0;
  for (int64_t bh = blockIdx.y; bh < bh_count; bh += gridDim.y) {
    const int64_t idx = bh * per_slab + i;
    uint4 x = k[idx];
    if (kRope && p.rot) x = rope_chunk(x, tab, pair0);
    kh[idx] = x;
    v16[idx] = bf16x8_to_f16x8(v[idx]);
  }
}

// ------------------------------------------------------------ fused attention

constexpr int kWaves = 8;
constexpr int kThreads = 64 * kWaves;
constexpr int BM = 32 * kWaves;  // query rows per workgroup (32 per wave)
constexpr int BN = 64;           // keys per tile
constexpr int KS = D + 8;        // K tile row stride in LDS (elements): 272 B
constexpr int VS = D + 32;       // V tile row stride in LDS (elements): 320 B
constexpr int kTabLdsPairs = 6144;  // rotary tables up to 48 KB are staged in LDS
constexpr float kLazyRescaleLog2 = 8.0f;
static_assert(kThreads == 8 * BN, "staging: one tile row per 8 threads, two 16-byte chunks each");

// Scheduling-group masks of __builtin_amdgcn_sched_group_barrier.
constexpr int kSgMfma = 0x008, kSgValu = 0x002, kSgDsRead = 0x100, kSgDsWrite = 0x200;

// First table pair of chunk c (< 8: frame or row axis) and c + 8 (row or column axis).
__device__ __forceinline__ int tab_pair_lo(int c, const Pos& p, const SeqGrid& g) {
  return c < 4 ? p.t * 16 + 4 * c : g.tab_h + p.h * 24 + 4 * (c - 4);
}
__device__ __forceinline__ int tab_pair_hi(int c, const Pos& p, const SeqGrid& g) {
  return c < 2 ? g.tab_h + p.h * 24 + 4 * (c + 4) : g.tab_w + p.w * 24 + 4 * (c - 2);
}

// Software pipeline, per wave, one barrier per 64-key tile.  Iteration i:
//   phase A (one scheduling region): S(i+1) = K^(i+1) Q^^T on the matrix
//     cores, interleaved with P(i) = exp2(S(i) c - m c) and its row sums on
//     the VALU -- independent work, so the two pipes overlap;
//   phase B (one region): O^T += V(i)^T P(i)^T on the matrix cores,
//     interleaved with staging K(i+2) (rotated, bf16) and V(i+1) (fp16) from
//     registers into LDS;
//   then the mask, row max and (rare) lazy rescale for tile i+1.
// K runs one tile ahead of V.  LDS: K(i+1) is read while K(i+2) is written
// over K(i) (last read in iteration i-1); V(i) is read while V(i+1) is
// written over V(i-1); the barrier ending each iteration orders every reuse.
// Loads past the last tile re-read row N-1 and land in buffers nobody reads,
// so phases A and B are branch-free.
// kRope: rotate Q (and K unless kPre) with the table; kTabLds: the table is
// staged in LDS; kPre: k is already rotated and v already fp16 (workspace
// path), so staging is a plain copy.
template <bool kRope, bool kTabLds, bool kPre>
__global__ __launch_bounds__(kThreads, 1) void attn_fwd_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
    const uint16_t* __restrict__ v, uint16_t* __restrict__ out, SeqGrid g,
    const float2* __restrict__ tab_g, int tab_pairs, int n_qtiles, float c_log2) {
  __shared__ __attribute__((aligned(16))) uint16_t k_lds[2][BN * KS];
  __shared__ __attribute__((aligned(16))) uint16_t v_lds[2][BN * VS];
  __shared__ __attribute__((aligned(16))) float2 tab_lds[kTabLds ? kTabLdsPairs : 2];

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

  const float2* tab = tab_g;
  if (kRope && kTabLds) {
    for (int i = tid * 2; i < tab_pairs; i += 2 * kThreads)  // tab_pairs is a multiple of 4
      *reinterpret_cast<float4*>(&tab_lds[i]) = *reinterpret_cast<const float4*>(&tab_g[i]);
    tab = tab_lds;
  }

  // ---- Q^ fragment (B operand of S^T = K^ Q^^T): dims [16kk + 8hh, +8) of one row.
  const int qrow = qt * BM + wave * 32 + l32;
  bf16x8 qf[8];
  {
    const uint4* src = reinterpret_cast<const uint4*>(qs + (size_t)min(qrow, N - 1) * D);
    Pos p{0, 0, 0, false};
    if (kRope) p = token_pos(min(qrow, N - 1), g);
    if (kRope && kTabLds) __syncthreads();  // table staged
#pragma unroll
    for (int kk = 0; kk < 8; ++kk) {
      const int cc = 2 * kk + hh;
      uint4 x = src[cc];
      // prefix tokens sit at (0, 0, 0): cos 0 = 1, sin 0 = 0, an exact identity
      if (kRope) x = rope_chunk(x, tab, tab_pair(cc, p, g));
      qf[kk] = __builtin_bit_cast(bf16x8, x);
    }
  }

  // ---- staging: thread moves chunks c0 and c0 + 8 of tile row rr.
  const int rr = tid >> 3;
  const int c0 = tid & 7;
  uint4 kreg[2], vreg[2];
  float4 kcs[4];  // (cos, sin) of the 8 rotary pairs of the two staged K chunks
  auto load_kv = [&](int kv0k, int kv0v) {
    const uint4* sk = reinterpret_cast<const uint4*>(ks + (size_t)min(kv0k + rr, N - 1) * D);
    const uint4* sv = reinterpret_cast<const uint4*>(vs + (size_t)min(kv0v + rr, N - 1) * D);
    kreg[0] = sk[c0];
    kreg[1] = sk[c0 + 8];
    vreg[0] = sv[c0];
    vreg[1] = sv[c0 + 8];
  };
  auto fetch_k_rotation = [&](int kv0) {
    if (kRope && !kPre) {
      const Pos p = token_pos(min(kv0 + rr, N - 1), g);
      const int a0 = tab_pair_lo(c0, p, g), a1 = tab_pair_hi(c0, p, g);
      kcs[0] = *reinterpret_cast<const float4*>(tab + a0);
      kcs[1] = *reinterpret_cast<const float4*>(tab + a0 + 2);
      kcs[2] = *reinterpret_cast<const float4*>(tab + a1);
      kcs[3] = *reinterpret_cast<const float4*>(tab + a1 + 2);
    }
  };
  auto store_k = [&](int buf) {
    uint4 x0 = kreg[0], x1 = kreg[1];
    if (kRope && !kPre) {
      x0 = rope_rotate(x0, kcs[0], kcs[1]);
      x1 = rope_rotate(x1, kcs[2], kcs[3]);
    }
    *reinterpret_cast<uint4*>(&k_lds[buf][rr * KS + c0 * 8]) = x0;
    *reinterpret_cast<uint4*>(&k_lds[buf][rr * KS + c0 * 8 + 64]) = x1;
  };
  auto store_v = [&](int buf) {
    *reinterpret_cast<uint4*>(&v_lds[buf][rr * VS + c0 * 8]) = kPre ? vreg[0] : bf16x8_to_f16x8(vreg[0]);
    *reinterpret_cast<uint4*>(&v_lds[buf][rr * VS + c0 * 8 + 64]) = kPre ? vreg[1] : bf16x8_to_f16x8(vreg[1]);
  };

  // K fragment (A operand) of key block kb (0/1), dims [16kk + 8hh, +8).
  auto kfrag = [&](const uint16_t* kbuf, int kb, int kk) {
    return *reinterpret_cast<const bf16x8*>(kbuf + (32 * kb + l32) * KS + kk * 16 + hh * 8);
  };
  auto scores = [&](int buf, f32x16& s0, f32x16& s1) {
    const uint16_t* kb = k_lds[buf];
    s0 = f32x16{};
    s1 = f32x16{};
#pragma unroll
    for (int kk = 0; kk < 8; ++kk) {
      s0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kfrag(kb, 0, kk), qf[kk], s0, 0, 0, 0);
      s1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kfrag(kb, 1, kk), qf[kk], s1, 0, 0, 0);
    }
  };

  // V^T operand addressing for the transpose read: within each 16-lane group,
  // lane 4s + c supplies row s (of 4) and 4 columns starting at 4c.
  const int g16 = lane >> 4, i16 = lane & 15;
  const int v_off = (4 * (g16 >> 1) + (i16 >> 2)) * VS + 16 * (g16 & 1) + 4 * (i16 & 3);

  f32x16 o[4];
#pragma unroll
  for (int db = 0; db < 4; ++db) o[db] = f32x16{};
  float m_run = -__builtin_inff();
  float l_run = 0.0f;
  const f16x2 ones = {(_Float16)1.0f, (_Float16)1.0f};

  // Mask keys >= N (tile `it` is the ragged last one) and fold the tile's row
  // max into the running max (lazy rescale of o and l).
  auto row_max = [&](int it, f32x16& s0, f32x16& s1) {
    const int kv0 = it * BN;
    // Register j of a score block holds key 8(j/4) + 4hh + (j%4) of that block.
    if (kv0 + BN > N) {
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const int key = kv0 + 8 * (j >> 2) + 4 * hh + (j & 3);
        if (key >= N) s0[j] = -__builtin_inff();
        if (key + 32 >= N) s1[j] = -__builtin_inff();
      }
    }
    // a chain of three-input maxima (v_max3_f32): one instruction per two scores
    float mx = fmaxf(s0[0], s1[0]);
#pragma unroll
    for (int j = 1; j < 16; ++j) mx = fmaxf(fmaxf(mx, s0[j]), s1[j]);
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float m_new = fmaxf(m_run, mx);
    if (__any((m_new - m_run) * c_log2 > kLazyRescaleLog2)) {
      const float alpha = __builtin_amdgcn_exp2f((m_run - m_new) * c_log2);
      m_run = m_new;
      l_run *= alpha;
#pragma unroll
      for (int db = 0; db < 4; ++db) o[db] *= alpha;
    }
  };

  const int n_kv = (N + BN - 1) / BN;
  auto iteration = [&](int it, f32x16& cs0, f32x16& cs1, f32x16& ns0, f32x16& ns1) {
    load_kv((it + 2) * BN, (it + 1) * BN);
    fetch_k_rotation((it + 2) * BN);
    __builtin_amdgcn_sched_barrier(0);  // issue the loads first: phase B consumes them
    // ---- phase A: S(it+1) on MFMA; P(it) and its row sums on VALU.
    {
      const uint16_t* kb = k_lds[(it + 1) & 1];
      ns0 = f32x16{};
      ns1 = f32x16{};
      const float mc = m_run * c_log2;
      // P in fp16 pairs: word w holds logits 2w and 2w+1 (s0[0..15] then s1[0..15])
      uint32_t pw[16];
      float la = 0.0f, lb = 0.0f;
#pragma unroll
      for (int kk = 0; kk < 8; ++kk) {
        ns0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kfrag(kb, 0, kk), qf[kk], ns0, 0, 0, 0);
        ns1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kfrag(kb, 1, kk), qf[kk], ns1, 0, 0, 0);
        // logits 4kk .. 4kk+3 of this lane
#pragma unroll
        for (int u = 0; u < 2; ++u) {
          const int idx = 4 * kk + 2 * u;
          const float a = idx < 16 ? cs0[idx] : cs1[idx - 16];
          const float b = idx < 16 ? cs0[idx + 1] : cs1[idx - 15];
          f16x2 h;
          h[0] = (_Float16)__builtin_amdgcn_exp2f(__builtin_fmaf(a, c_log2, -mc));
          h[1] = (_Float16)__builtin_amdgcn_exp2f(__builtin_fmaf(b, c_log2, -mc));
          pw[2 * kk + u] = __builtin_bit_cast(uint32_t, h);
        }
        // row sums of the rounded probabilities (exact fp32 sums of fp16
        // values), so numerator and denominator weigh keys identically
        la = __builtin_amdgcn_fdot2(__builtin_bit_cast(f16x2, pw[2 * kk]), ones, la, false);
        lb = __builtin_amdgcn_fdot2(__builtin_bit_cast(f16x2, pw[2 * kk + 1]), ones, lb, false);
      }
      f16x8 pb[4];
#pragma unroll
      for (int t = 0; t < 4; ++t)
        pb[t] = __builtin_bit_cast(f16x8, make_uint4(pw[4 * t], pw[4 * t + 1], pw[4 * t + 2], pw[4 * t + 3]));
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        __builtin_amdgcn_sched_group_barrier(kSgDsRead, 2, 0);
        __builtin_amdgcn_sched_group_barrier(kSgMfma, 2, 0);
        __builtin_amdgcn_sched_group_barrier(kSgValu, 12, 0);
      }
      l_run += la + lb;
      // ---- phase B: O^T += V(it)^T P(it)^T on MFMA; staging on VALU.
      const uint16_t* vb = v_lds[it & 1] + v_off;
#pragma unroll
      for (int kst = 0; kst < 4; ++kst) {
#pragma unroll
        for (int db = 0; db < 4; ++db) {
          const uint16_t* p0 = vb + 16 * kst * VS + 32 * db;
          const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)p0);
          const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p0 + 8 * VS));
          const f16x8 a = __builtin_bit_cast(
              f16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
          o[db] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, pb[kst], o[db], 0, 0, 0);
        }
      }
      store_k(it & 1);
      store_v((it + 1) & 1);
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        __builtin_amdgcn_sched_group_barrier(kSgDsRead, 2, 1);
        __builtin_amdgcn_sched_group_barrier(kSgMfma, 1, 1);
        __builtin_amdgcn_sched_group_barrier(kSgValu, 6, 1);
      }
      __builtin_amdgcn_sched_group_barrier(kSgDsWrite, 4, 1);
    }
    if (it + 1 < n_kv) row_max(it + 1, ns0, ns1);
    __syncthreads();
  };

  // ---- prologue: K(0), V(0), K(1) into LDS; S(0) and its row max.
  load_kv(0, 0);
  fetch_k_rotation(0);
  store_k(0);
  store_v(0);
  load_kv(BN, BN);
  fetch_k_rotation(BN);
  store_k(1);
  __syncthreads();
  f32x16 sa0, sa1, sb0, sb1;
  scores(0, sa0, sa1);
  row_max(0, sa0, sa1);
  __syncthreads();  // K(2) will overwrite K(0)

  int it = 0;
  for (; it + 1 < n_kv; it += 2) {
    iteration(it, sa0, sa1, sb0, sb1);
    iteration(it + 1, sb0, sb1, sa0, sa1);
  }
  if (it < n_kv) iteration(it, sa0, sa1, sb0, sb1);

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
  const int tab_pairs = g.tab_w + g.Wl * (3 * D / 16);
  if (tab == nullptr)
    hipLaunchKernelGGL((attn_fwd_kernel<false, false, false>), grid, dim3(kThreads), 0, stream, q,
                       k, v, out, g, tab, 0, n_qtiles, c_log2);
  else if (tab_pairs <= kTabLdsPairs)
    hipLaunchKernelGGL((attn_fwd_kernel<true, true, false>), grid, dim3(kThreads), 0, stream, q,
                       k, v, out, g, tab, tab_pairs, n_qtiles, c_log2);
  else
    hipLaunchKernelGGL((attn_fwd_kernel<true, false, false>), grid, dim3(kThreads), 0, stream, q,
                       k, v, out, g, tab, tab_pairs, n_qtiles, c_log2);
  return hipGetLastError();
}

hipError_t launch_prepare_kv(const uint16_t* k, const uint16_t* v, uint16_t* k_rot,
                             uint16_t* v_f16, int BH, const SeqGrid& g, const float2* tab,
                             hipStream_t stream) {
  const int64_t per_slab = (int64_t)g.n * kChunks;
  const dim3 pgrid((unsigned)((per_slab + 255) / 256), (unsigned)(BH < 65535 ? BH : 65535));
  if (tab != nullptr)
    hipLaunchKernelGGL(prep_kv_kernel<true>, pgrid, dim3(256), 0, stream,
                       reinterpret_cast<const uint4*>(k), reinterpret_cast<const uint4*>(v),
                       reinterpret_cast<uint4*>(k_rot), reinterpret_cast<uint4*>(v_f16),
                       (int64_t)BH, g, tab);
  else
    hipLaunchKernelGGL(prep_kv_kernel<false>, pgrid, dim3(256), 0, stream,
                       reinterpret_cast<const uint4*>(k), reinterpret_cast<const uint4*>(v),
                       reinterpret_cast<uint4*>(k_rot), reinterpret_cast<uint4*>(v_f16),
                       (int64_t)BH, g, tab);
  return hipGetLastError();
}

hipError_t launch_attn_fwd_prepared(const uint16_t* q, const uint16_t* k_rot,
                                    const uint16_t* v_f16, uint16_t* out, int BH,
                                    const SeqGrid& g, const float2* tab, hipStream_t stream) {
  const int n_qtiles = (g.n + BM - 1) / BM;
  const float c_log2 = (float)(1.4426950408889634 / 11.313708498984761);  // log2(e)/sqrt(128)
  const dim3 grid((unsigned)((int64_t)n_qtiles * BH));
  if (tab != nullptr)
    hipLaunchKernelGGL((attn_fwd_kernel<true, false, true>), grid, dim3(kThreads), 0, stream, q,
                       k_rot, v_f16, out, g, tab, 0, n_qtiles, c_log2);
  else
    hipLaunchKernelGGL((attn_fwd_kernel<false, false, true>), grid, dim3(kThreads), 0, stream, q,
                       k_rot, v_f16, out, g, tab, 0, n_qtiles, c_log2);
  return hipGetLastError();
}

int64_t attn_max_workgroups(int N, int BH) { return (int64_t)((N + BM - 1) / BM) * BH; }

}  // namespace sol
