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
#include <mutex>

#include "sol_device.h"

namespace sol {
namespace {

// ------------------------------------------------------------ range status

// Sticky range status of the device, read by sol_range_status: bits the
// kernels set when a converted fp16 operand of the prepared path (q', k^, v)
// or an output element is not finite.  Zero when the library is loaded.
__device__ unsigned range_flags;

// The tests below read the bits of floating-point values.  The library is
// built with -fno-honor-nans, under which the compiler turns a test of the
// exponent bits back into a floating-point compare with infinity that
// assumes NaN away; the empty asm hides the bits' origin from it.
__device__ __forceinline__ uint32_t opaque_bits(uint32_t u) {
  asm volatile("" : "+v"(u));
  return u;
}
// Any of the eight fp16 values of x is inf or NaN (exponent field all ones).
__device__ __forceinline__ bool f16x8_nonfinite(uint4 x) {
  const uint32_t w[4] = {x.x, x.y, x.z, x.w};
  bool bad = false;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const uint32_t m = opaque_bits(w[u]) & 0x7C007C00u;
    bad |= (m & 0xFFFFu) == 0x7C00u || (m >> 16) == 0x7C00u;
  }
  return bad;
}
// x is inf or NaN (exponent field all ones).
__device__ __forceinline__ bool f32_nonfinite(float x) {
  return (opaque_bits(__float_as_uint(x)) & 0x7F800000u) == 0x7F800000u;
}
// One atomic per wave in which some lane saw a bad value.
__device__ __forceinline__ void note_range(bool bad, unsigned flag) {
  const uint64_t m = __ballot(bad);
  if (m != 0 && __lane_id() == (unsigned)__builtin_ctzll(m)) atomicOr(&range_flags, flag);
}

// --------------------------------------------------------- standalone rotary

// One thread per 16-byte chunk of one (b, h) slab; grid.y walks the slabs.
// gamma != NULL: each row is RMS-normalised first (the 16 chunks of a row sit
// in 16 consecutive lanes; rows are never split across waves).
__global__ __launch_bounds__(256) void rope3d_kernel(const uint4* __restrict__ x,
                                                     uint4* __restrict__ y, int64_t bh_count,
                                                     SeqGrid g, const float2* __restrict__ tab,
                                                     const float* __restrict__ gamma, float eps) {
  const int64_t per_slab = (int64_t)g.n * kChunks;
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= per_slab) return;  // whole rows: the lanes of a row leave together
  const int n = (int)(i / kChunks);
  const int cc = (int)(i % kChunks);
  const Pos p = token_pos(n, g);
  const bool rot = p.rot && tab != nullptr;
  const int pair0 = rot ? tab_pair(cc, p, g) : 0;
  for (int64_t bh = blockIdx.y; bh < bh_count; bh += gridDim.y) {
    const int64_t idx = bh * per_slab + i;
    const uint4 v = x[idx];
    const float inv = gamma ? rms_inv(row_sumsq_lanes16(chunk_sumsq(v)), eps) : 1.0f;
    y[idx] = qk_chunk(v, gamma, inv, cc, rot, tab, tab_lo_plane(tab, g), pair0);
  }
}

// Prepared K/V for the prepared-path kernel: per (b, h) slab and 32-key tile,
// 8 KB of K and 8 KB of V, each laid out in the order the kernel's MFMA
// fragments are read, so one tile is one contiguous copy into LDS and every
// fragment read is one linear ds_read_b128 (64 lanes x 16 bytes, no bank
// conflicts, immediate offsets).
//   K tile: [kk 0..7][lane 0..63][8]: lane = r + 32 hh holds K^[key r][16kk + 8hh ..+7],
//     K^ the rotated (and, with gamma, first normalised) key rounded to bf16
//     (as every rotation here), then fp16.
//   V tile: [j 0..7][lane 0..63][8], j = 4 kst + db: lane = l + 32 hh holds
//     V[key 16kst + 8(i/4) + 4hh + i%4][dim 32db + l] for i = 0..7, fp16 -- the
//     key order of the fp16 probability words the PV MFMA multiplies it with.
// The source holds g.n keys per slab; they land at keys key0 .. key0 + g.n - 1
// of a prepared sequence of n_kv keys (several calls fill one sequence from
// several sources, e.g. cached reference keys and the current step's).  Keys
// past n_kv are zero.  A tile that also holds keys of another source is
// written element by element, only where this call owns the key.  One
// workgroup per tile (from tile0 on); grid.y walks the slabs.

template <bool kRope, bool kRec>
__global__ __launch_bounds__(256) void prep_kv_kernel(const uint4* __restrict__ k,
                                                      const uint4* __restrict__ v,
                                                      uint4* __restrict__ kp, uint4* __restrict__ vp,
                                                      int64_t bh_count, SeqGrid g,
                                                      const float2* __restrict__ tab, int key0,
                                                      int n_kv, int tile0,
                                                      const float* __restrict__ gamma, float eps,
                                                      const uint8_t* __restrict__ rec, int heads) {
  __shared__ __attribute__((aligned(16))) uint16_t vt[kPrepTile * (D + 8)];
  lds_poison(vt, sizeof(vt));
  lds_poison_done();
  const float2* __restrict__ tab_lo = tab_lo_plane(tab, g);
  const int n_src = g.n;
  const int n_tiles = (n_kv + kPrepTile - 1) / kPrepTile;  // tiles per prepared slab
  const int tile = tile0 + blockIdx.x;
  const int t = threadIdx.x;
  const int first = tile * kPrepTile;
  // Key dst of this tile is written by this call when it is one of its own
  // (key0 <= dst < key0 + n_src) or padding past the sequence (dst >= n_kv).
  auto owned = [&](int dst) { return (dst >= key0 && dst - key0 < n_src) || dst >= n_kv; };
  const bool whole = first >= key0 && min(first + kPrepTile, n_kv) <= key0 + n_src;
  // This thread's two 16-byte chunks of the tile: row r, chunk cc (dims 8cc..8cc+7).
  int r[2], cc[2], pair0[2], src[2];
  bool valid[2], rot[2];
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int c = t + 256 * u;
    r[u] = c >> 4;
    cc[u] = c & 15;
    src[u] = first + r[u] - key0;
    valid[u] = src[u] >= 0 && src[u] < n_src;
    Pos p{0, 0, 0, false};
    if (kRope && valid[u]) p = token_pos(src[u], g);
    rot[u] = kRope && p.rot;
    pair0[u] = rot[u] ? tab_pair(cc[u], p, g) : 0;
  }
  const uint4 zero = make_uint4(0u, 0u, 0u, 0u);
  bool bad_k = false, bad_v = false;  // an fp16 operand out of range (or not finite)
  for (int64_t bh = blockIdx.y; bh < bh_count; bh += gridDim.y) {
    const size_t row0 = (size_t)bh * n_src;
    uint4* kt = kp + ((size_t)bh * n_tiles + tile) * (kPrepTileElems / 8);
    uint4* vtile = vp + ((size_t)bh * n_tiles + tile) * (kPrepTileElems / 8);
    // kRec: the keys and values come decoded from the block-INT8 records of
    // the (b, h) slab, token-major with `heads` records per token
    const int64_t rb = kRec ? bh / heads : 0;
    const size_t rslab = kRec ? (size_t)rb * n_src * heads + (size_t)(bh - rb * heads) : 0;
    auto rec_of = [&](int u) { return rec + (rslab + (size_t)src[u] * heads) * kRecBytes; };
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      if (kRec) {
        // records carry k as attention consumes it (normalised and rotated)
        const uint4 xr = valid[u] ? rec_chunk(rec_of(u), 1, cc[u]) : zero;
        const uint4 xh = bf16x8_to_f16x8(xr);
        bad_k |= f16x8_nonfinite(xh);
        if (owned(first + r[u])) kt[(cc[u] >> 1) * 64 + r[u] + 32 * (cc[u] & 1)] = xh;
      } else {
        const uint4 x = valid[u] ? k[(row0 + src[u]) * kChunks + cc[u]] : zero;
        // every lane takes part in the row sums (rows sit in 16 aligned lanes)
        const float inv = gamma ? rms_inv(row_sumsq_lanes16(chunk_sumsq(x)), eps) : 1.0f;
        const uint4 xr = valid[u] ? qk_chunk(x, gamma, inv, cc[u], rot[u], tab, tab_lo, pair0[u]) : zero;
        const uint4 xh = bf16x8_to_f16x8(xr);
        bad_k |= f16x8_nonfinite(xh);
        if (owned(first + r[u])) kt[(cc[u] >> 1) * 64 + r[u] + 32 * (cc[u] & 1)] = xh;
      }
      const uint4 y = !valid[u] ? zero
                      : kRec    ? rec_chunk(rec_of(u), 2, cc[u])
                                : v[(row0 + src[u]) * kChunks + cc[u]];
      const uint4 yh = bf16x8_to_f16x8(y);
      bad_v |= f16x8_nonfinite(yh);
      *reinterpret_cast<uint4*>(&vt[r[u] * (D + 8) + cc[u] * 8]) = yh;
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int c = t + 256 * u;
      const int j = c >> 6, ln = c & 63;
      const int kst = j >> 2, db = j & 3, l = ln & 31, h = ln >> 5;
      const uint16_t* col = vt + (16 * kst + 4 * h) * (D + 8) + 32 * db + l;
      auto key = [&](int i) { return 16 * kst + 4 * h + 8 * (i >> 2) + (i & 3); };
      auto el = [&](int i) { return (uint32_t)col[(8 * (i >> 2) + (i & 3)) * (D + 8)]; };
      if (whole) {
        vtile[c] = make_uint4(el(0) | el(1) << 16, el(2) | el(3) << 16, el(4) | el(5) << 16,
                              el(6) | el(7) << 16);
      } else {
        uint16_t* dst = reinterpret_cast<uint16_t*>(vtile + c);
#pragma unroll
        for (int i = 0; i < 8; ++i)
          if (owned(first + key(i))) dst[i] = (uint16_t)el(i);
      }
    }
    __syncthreads();
  }
  note_range(bad_k, SOL_RANGE_K);
  note_range(bad_v, SOL_RANGE_V);
}

// ------------------------------------------------------------ fused attention

constexpr int kWaves = 8;
constexpr int kThreads = 64 * kWaves;
constexpr int BM = 32 * kWaves;  // query rows per workgroup (32 per wave)
static_assert(BM == kFusedRows, "the host sizes the fused grid with kFusedRows");
constexpr int BN = 64;           // keys per tile
constexpr int KS = D + 8;        // K tile row stride in LDS (elements): 272 B
constexpr int VS = D + 32;       // V tile row stride in LDS (elements): 320 B
constexpr int kTabLdsPairs = 6144;  // rotary tables up to 48 KB are staged in LDS
// A tile's probabilities are taken against the running reference max m; they
// stay finite in fp16 while they do not exceed 2^15 (fp16 max 65504).  A
// lane's fp32 sum over its 32 probabilities bounds each of them, so the sum
// (needed anyway) doubles as the overflow check; only when it exceeds 2^15 is
// the tile's own max folded into m (rare: once the first tiles have set m).
constexpr float kP16SumLimit = 32768.0f;
static_assert(kThreads == 8 * BN, "staging: one tile row per 8 threads, two 16-byte chunks each");

// Scheduling-group masks of __builtin_amdgcn_sched_group_barrier.
constexpr int kSgMfma = 0x008, kSgValu = 0x002, kSgDsRead = 0x100, kSgDsWrite = 0x200;

// First table pair of chunk c (< 8: frame or row axis) and c + 8 (row or column
// axis) under the default 32/48/48 split -- the only one sol_attn_fwd, whose
// signature carries no split, launches this kernel with -- in two selects
// instead of tab_pair's three.
__device__ __forceinline__ int tab_pair_lo(int c, const Pos& p, const SeqGrid& g) {
  return c < 4 ? p.t * 16 + 4 * c : g.tab_h + p.h * 24 + 4 * (c - 4);
}
__device__ __forceinline__ int tab_pair_hi(int c, const Pos& p, const SeqGrid& g) {
  return c < 2 ? g.tab_h + p.h * 24 + 4 * (c + 4) : g.tab_w + p.w * 24 + 4 * (c - 2);
}
static_assert(kSplitT == 32 && kSplitH == 48 && kSplitW == 48, "tab_pair_lo/hi assume 32/48/48");

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
// kRope: rotate Q and K with the table; kTabLds: the table is staged in LDS.
template <bool kRope, bool kTabLds>
__global__ __launch_bounds__(kThreads, 1) void attn_fwd_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
    const uint16_t* __restrict__ v, uint16_t* __restrict__ out, SeqGrid g,
    const float2* __restrict__ tab_g, int tab_pairs, int n_qtiles, float c_log2) {
  __shared__ __attribute__((aligned(16))) uint16_t k_lds[2][BN * KS];
  __shared__ __attribute__((aligned(16))) uint16_t v_lds[2][BN * VS];
  __shared__ __attribute__((aligned(16))) float2 tab_lds[kTabLds ? kTabLdsPairs : 2];
  lds_poison(k_lds, sizeof(k_lds));
  lds_poison(v_lds, sizeof(v_lds));
  lds_poison(tab_lds, sizeof(tab_lds));
  lds_poison_done();

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
  // queries turn exactly (both planes, from global memory: once per workgroup);
  // key tiles turn in fp32 with the hi plane, staged in LDS when it fits
  const float2* tab_lo = kRope ? tab_g + tab_pairs : nullptr;
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
      if (kRope) x = rope_chunk(x, tab, tab_lo, tab_pair(cc, p, g));
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
    if (kRope) {
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
    if (kRope) {
      x0 = rope_rotate_fast(x0, kcs[0], kcs[1]);
      x1 = rope_rotate_fast(x1, kcs[2], kcs[3]);
    }
    *reinterpret_cast<uint4*>(&k_lds[buf][rr * KS + c0 * 8]) = x0;
    *reinterpret_cast<uint4*>(&k_lds[buf][rr * KS + c0 * 8 + 64]) = x1;
  };
  auto store_v = [&](int buf) {
    *reinterpret_cast<uint4*>(&v_lds[buf][rr * VS + c0 * 8]) = bf16x8_to_f16x8(vreg[0]);
    *reinterpret_cast<uint4*>(&v_lds[buf][rr * VS + c0 * 8 + 64]) = bf16x8_to_f16x8(vreg[1]);
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

  // Keys >= N get no weight (tile `it` is the ragged last one).
  auto mask_tile = [&](int it, f32x16& s0, f32x16& s1) {
    const int kv0 = it * BN;
    // Register j of a score block holds key 8(j/4) + 4hh + (j%4) of that block.
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const int key = kv0 + 8 * (j >> 2) + 4 * hh + (j & 3);
      if (key >= N) s0[j] = -__builtin_inff();
      if (key + 32 >= N) s1[j] = -__builtin_inff();
    }
  };
  // Fold a tile's row max into the reference max m, rescaling o and l.
  auto fold_max = [&](const f32x16& s0, const f32x16& s1) {
    // a chain of three-input maxima (v_max3_f32): one instruction per two scores
    float mx = fmaxf(s0[0], s1[0]);
#pragma unroll
    for (int j = 1; j < 16; ++j) mx = fmaxf(fmaxf(mx, s0[j]), s1[j]);
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float m_new = fmaxf(m_run, mx);
    const float alpha = __builtin_amdgcn_exp2f((m_run - m_new) * c_log2);  // 0 for the first tile
    m_run = m_new;
    l_run *= alpha;
#pragma unroll
    for (int db = 0; db < 4; ++db) o[db] *= alpha;
  };
  // fp16 probabilities of one tile against m (word w: logits 2w, 2w+1 of
  // s0[0..15] then s1[0..15]) and their per-lane sum.
  auto probs = [&](const f32x16& s0, const f32x16& s1, uint32_t* pw, float& la, float& lb) {
    const float mc = m_run * c_log2;
    la = 0.0f;
    lb = 0.0f;
#pragma unroll
    for (int w = 0; w < 16; ++w) {
      const float a = w < 8 ? s0[2 * w] : s1[2 * w - 16];
      const float b = w < 8 ? s0[2 * w + 1] : s1[2 * w - 15];
      const float ea = __builtin_amdgcn_exp2f(__builtin_fmaf(a, c_log2, -mc));
      const float eb = __builtin_amdgcn_exp2f(__builtin_fmaf(b, c_log2, -mc));
      f16x2 h;
      h[0] = (_Float16)ea;
      h[1] = (_Float16)eb;
      pw[w] = __builtin_bit_cast(uint32_t, h);
      la += ea;
      lb += eb;
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
          const float ea = __builtin_amdgcn_exp2f(__builtin_fmaf(a, c_log2, -mc));
          const float eb = __builtin_amdgcn_exp2f(__builtin_fmaf(b, c_log2, -mc));
          f16x2 h;
          h[0] = (_Float16)ea;
          h[1] = (_Float16)eb;
          pw[2 * kk + u] = __builtin_bit_cast(uint32_t, h);
          // row sums in fp32 adds: v_dot2_f32_f16 would share the matrix
          // pipe with the MFMAs and cost about half an MFMA each
          la += ea;
          lb += eb;
        }
      }
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        __builtin_amdgcn_sched_group_barrier(kSgDsRead, 2, 0);
        __builtin_amdgcn_sched_group_barrier(kSgMfma, 2, 0);
        __builtin_amdgcn_sched_group_barrier(kSgValu, 12, 0);
      }
      if (__any(la + lb > kP16SumLimit)) {  // rare: m lags this tile by > 2^15
        fold_max(cs0, cs1);
        probs(cs0, cs1, pw, la, lb);
      }
      l_run += la + lb;
      f16x8 pb[4];
#pragma unroll
      for (int t = 0; t < 4; ++t)
        pb[t] = __builtin_bit_cast(f16x8, make_uint4(pw[4 * t], pw[4 * t + 1], pw[4 * t + 2], pw[4 * t + 3]));
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
    if (it + 1 < n_kv && (it + 2) * BN > N) mask_tile(it + 1, ns0, ns1);
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
  if (BN > N) mask_tile(0, sa0, sa1);
  fold_max(sa0, sa1);  // the first tile sets the reference max
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
  {
    // an output that is not finite is reported (|v| >= 65504 overflows the
    // fp16 value operand; inf or NaN inputs): an inf or NaN accumulator, or
    // 1/l, makes the lane's sum of them inf or NaN
    float sum = inv;
#pragma unroll
    for (int db = 0; db < 4; ++db)
#pragma unroll
      for (int j = 0; j < 16; ++j) sum += o[db][j];
    note_range(f32_nonfinite(sum) && qrow < N, SOL_RANGE_OUT);
  }
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

// ------------------------------------------------- attention on prepared K/V

// bf16 x8 -> fp32, times s (fp32, RNE) -> fp16 x8 (RNE).
__device__ __forceinline__ f16x8 bf16x8_to_f16x8_scaled(uint4 x, float s) {
  const uint32_t w[4] = {x.x, x.y, x.z, x.w};
  f16x8 r;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    r[2 * u] = (_Float16)(__uint_as_float(w[u] << 16) * s);
    r[2 * u + 1] = (_Float16)(__uint_as_float(w[u] & 0xffff0000u) * s);
  }
  return r;
}

// Score MFMAs as inline assembly: the result goes to VGPRs, where the softmax
// reads it, while the query operand stays in AGPRs (the builtin would put the
// result in AGPRs, next to the output accumulators, and every score would
// cost a v_accvgpr_read).  The compiler does not see these as MFMAs, so every
// VALU access to their results or their srcC is placed after mfma_wait() or
// far behind them (the next iteration).
__device__ __forceinline__ void mfma_s_first(f32x16& d, const f16x8& k, const f16x8& q,
                                             const f32x16& c) {
  asm volatile("v_mfma_f32_32x32x16_f16 %0, %1, %2, %3" : "=&v"(d) : "v"(k), "a"(q), "v"(c));
}
__device__ __forceinline__ void mfma_s_next(f32x16& d, const f16x8& k, const f16x8& q) {
  asm volatile("v_mfma_f32_32x32x16_f16 %0, %1, %2, %0" : "+v"(d) : "v"(k), "a"(q));
}
// 16 wait states: more than the 12 an 8-pass MFMA result needs before the VALU
// reads or overwrites it.
__device__ __forceinline__ void mfma_wait() { asm volatile("s_nop 7\n\ts_nop 7" ::: "memory"); }
// 4 wait states, after a dozen independent instructions have already issued.
__device__ __forceinline__ void mfma_wait_tail() { asm volatile("s_nop 3" ::: "memory"); }
// Two fp32 values as an fp16 pair (RNE), the low half first.
__device__ __forceinline__ uint32_t pack_f16x2(float lo, float hi) {
  f16x2 h;
  h[0] = (_Float16)lo;
  h[1] = (_Float16)hi;
  return __builtin_bit_cast(uint32_t, h);
}
// Sum of two fp16 pairs, lane-wise (v_pk_add_f16).
__device__ __forceinline__ uint32_t add_f16x2(uint32_t a, uint32_t b) {
  return __builtin_bit_cast(uint32_t, __builtin_bit_cast(f16x2, a) + __builtin_bit_cast(f16x2, b));
}
// The two halves of an fp16 pair added in fp32.
__device__ __forceinline__ float sum_f16x2(uint32_t a) {
  const f16x2 h = __builtin_bit_cast(f16x2, a);
  return (float)h[0] + (float)h[1];
}
// Keep a value computed where it stands: IR passes would otherwise sink the
// softmax arithmetic of a chunk to its first use and undo the interleaving.
__device__ __forceinline__ void pin(uint32_t& x) { asm volatile("" : "+v"(x)); }
__device__ __forceinline__ void pin(float& x) { asm volatile("" : "+v"(x)); }

// fp32 -> FP8 E4M3 code (the OCP E4M3FN format: bias 7, 3 mantissa bits, no
// infinities, 0x7F NaN), round to nearest even, saturating at +-448
// (infinities too).  The raw E4M3 output the paper's attention hands to the
// next GEMM with unit scales (Sec. 3.3, "Joint optimization with quantized
// communication").  Normal results keep 3 of fp32's 23 mantissa bits by an
// integer round-to-nearest-even on the bit pattern, then move the exponent
// from fp32's bias 127 to 7; below 2^-6 the quantum is fixed at 2^-9.
__device__ __forceinline__ uint32_t f32_to_e4m3(float x) {
  const uint32_t sign = (__float_as_uint(x) >> 24) & 0x80u;
  const float a = __builtin_fabsf(x);
  // NaN by its bits: the library is built with -fno-honor-nans
  if ((__float_as_uint(x) & 0x7FFFFFFFu) > 0x7F800000u) return 0x7Fu;
  if (a >= 448.0f) return sign | 0x7Eu;
  if (a < 0.015625f) return sign | (uint32_t)__builtin_rintf(a * 512.0f);  // 0..8, exact product
  const uint32_t ua = __float_as_uint(a);
  const uint32_t r = (ua + 0x7FFFFu + ((ua >> 20) & 1u)) >> 20;  // exponent:mantissa, rounded
  return sign | (r - (120u << 3));
}

// End of a prepared-path iteration: all but the last four vector-memory
// operations of this wave (this iteration's tile copies into LDS) complete,
// then the workgroup barrier -- after which every wave's completed copies are
// visible.  No LDS read needs to complete first: the next iteration's copies
// overwrite tiles whose fragments every wave read (and waited for) at least
// one iteration earlier.  The count of four holds only because the compiler
// issues no memory instruction of its own in the loop (no loads, stores or
// spills: a build test checks the generated code).
// kInflight: iterations whose copies may still be in flight (the dense walk
// 1; the block-sparse walk, whose scattered tiles miss L2 more often, 3: its
// copies are issued two iterations earlier).
template <int kInflight>
__device__ __forceinline__ void dma_barrier() {
  static_assert(kInflight >= 1 && kInflight <= 3, "vmcnt holds at most 15 here");
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0x0F70 | (4 * kInflight));  // vmcnt 4 kInflight, no LDS wait
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Attention on prepared K/V: k holds the rotated keys and v the values, both
// as fp16.  The query rows are rotated and rounded to bf16 like every rotation
// here, then multiplied by c = log2(e)/sqrt(D) and rounded to fp16, so the
// score MFMAs (fp16 x fp16 -> fp32) deliver c q.k.  Each chain of score MFMAs
// starts from a tile holding -m, the running reference max in those units, so
// the accumulator already holds the base-2 exponent of the softmax numerator
// (Eq. 1 with the 1/sqrt(D) scale; the online max of the flash formulation)
// and one probability costs a single v_exp_f32.
//
// 64 query rows per wave: every K fragment and V^T fragment read from LDS
// feeds two MFMAs (one per 32-query block).  4 waves (one per SIMD, 256 query
// rows per workgroup), the 2 x 4 output accumulators and Q' in AGPRs, 32-key
// tiles so that the scores of two tiles fit in VGPRs.  With one wave per SIMD
// the wave issues in order and nothing hides a stall, so each iteration i is
// laid out by hand in slots of ONE MFMA followed by the VALU and memory work
// that runs in its shadow (sched_barrier fences keep the order; two MFMAs in a
// row would leave the first one's shadow empty):
//   phase A: S(i+1) = K(i+1) Q'^T - m (16 MFMAs) beside the qb1 half of
//     P(i) = exp2(S(i)), and the reads of K(i+2) into the K fragment
//     registers as each fragment of K(i+1) is used;
//   phase B: O^T += V(i)^T P(i)^T (16 MFMAs) beside the qb0 half of P(i+1),
//     the reads of V(i+1) into the V fragment registers, and the copies of
//     K(i+4) and V(i+3) into LDS (one 1 KB block in each of four slots).
// Each pair of slots packs the previous pair's two probabilities (software
// pipelined: an exponential is never read by the very next instruction).  A
// row sum is the sum of the fp16 words themselves -- the very probabilities
// the PV MFMAs multiply -- added as fp16 pairs in a tree of seven
// v_pk_add_f16 per block and tile, then in fp32 across tiles.
// LDS holds rings of eight K tiles and four V tiles (96 KB); the barrier that
// ends an iteration waits only for the copies issued one iteration earlier.
constexpr int BN2 = kPrepTile;         // keys per tile of the prepared-path kernel
constexpr int kWaves2 = 4;             // waves per workgroup of the prepared-path kernel
constexpr int kKBufs = 8;              // K tiles in LDS (a power of two: ring
constexpr int kVBufs = 4;              // V tiles in LDS  offsets are masks)
// Descriptor word 3 of a raw buffer resource (32-bit data, no format swizzle).
constexpr int kBufferDword3 = 0x00020000;

// kSparse: block-sparse attention (Sec. 3.4, "Per-step dynamic sparsity").
// The workgroup's 256 query rows are one routing query block; it attends only
// to the key blocks (kSparseKeyBlock keys = 4 tiles each) listed for it in
// blocks[(bh * n_qtiles + qt) * nkb ..] (ascending, counts[bh * n_qtiles + qt]
// of them).  The list is staged into LDS once, each word holding an entry and
// the next one of the walk (ascending from the first entry);
// the loop walks the listed tiles in that order -- LDS ring slots follow the
// walk, copies read the listed tile.  One LDS read per iteration,
// issued at its start and made scalar halfway through phase A, gives the tiles of both
// copies (walk positions i + kVAhead and i + kKAhead lie in one block or two neighbours);
// masks need no lookup, since only the last listed block can hold keys past
// N and its walk position is known.
static_assert(kSparseQueryBlock == BM, "a routing query block is one workgroup's rows");

// kOutRec: block-INT8 output records (out_format 2), a template flag so that
// the bf16 and E4M3 instances do not carry the record epilogue's registers.
//
// Two launches.  Each row's reference max m starts at the largest score of
// the walk's first key tile and of the rows' diagonal tile.  The first launch
// (kRobust false) keeps m fixed: its loop carries no per-tile branch.  A wave
// whose probabilities leave the fp16 range against m (a score more than 15
// above it) stops computing at the end of that loop trip -- it keeps issuing
// its share of the tile copies and barriers for the other waves -- and writes
// its rows as NaN.  The second launch (kRobust true) recomputes exactly the
// row blocks so marked (every other workgroup leaves at once): there a tile
// whose probabilities would overflow raises m in place, while its scores are
// still in registers -- O and l rescaled -- before its probabilities are used.
// Neither kernel spills.  Exact softmax whatever the score distribution.
template <bool kRope, bool kRobust, bool kSparse, bool kRec, bool kOutRec>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1)))
void attn_prepared_kernel(const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
                          const uint16_t* __restrict__ v, uint16_t* __restrict__ out, SeqGrid g,
                          const float2* __restrict__ tab, int n_qtiles, float c_log2, int n_keys,
                          const float* __restrict__ q_gamma, float eps, int out_format,
                          const uint16_t* __restrict__ blocks, const int* __restrict__ counts,
                          int nkb, const uint8_t* __restrict__ qrec, int heads) {
  __shared__ __attribute__((aligned(1024))) uint16_t k_lds[kKBufs * kPrepTileElems];
  // The sparse walk copies K 6 and V 5 walk positions ahead (the dense walk
  // 4 and 3), with a V ring of 8: 64 + 64 + 32 KB, the whole 160 KB of LDS.
  // K(t) is read in iteration t - 2 and V(t) in t - 1, so the copies of the
  // last kInflight iterations may be in flight at an iteration's end.  (Three
  // iterations in flight measured 0.3-0.6 % faster than two, whose misses the
  // memory-side cache serves in the slab-synchronous order.)
  constexpr int kVB = kSparse ? 8 : kVBufs;
  constexpr int kKAhead = kSparse ? 6 : 4, kVAhead = kKAhead - 1;
  constexpr int kInflight = kKAhead - 3;
  static_assert(kKAhead <= 7 && kVAhead <= 7 && (kSparse || kVAhead <= 3),
                "a copy must land a barrier after the last read of the slot it overwrites");
  __shared__ __attribute__((aligned(1024))) uint16_t v_lds[kVB * kPrepTileElems];
  __shared__ uint32_t blist[kSparse ? kMaxSparseBlocks : 1];  // entry e | entry e + 1 << 16
  __shared__ int n_gave_up;  // first pass: waves of the workgroup that stopped computing
  lds_poison(k_lds, sizeof(k_lds));
  lds_poison(v_lds, sizeof(v_lds));
  lds_poison_done();

  auto keep = [&](auto& x) __attribute__((always_inline)) { pin(x); };
  // Score units.  First pass: q' = fp16(q^ c), c = log2(e)/sqrt(D), so the
  // score MFMAs return c q^.k^ and an exponential takes the accumulator as it
  // is.  q^ c rounded to fp16 carries a relative error of 2^-12 per element,
  // which moves a score by about 2^-12 of its size: negligible for the scores
  // of diffuse rows, but the rows the second pass takes are the peaked ones,
  // whose large scores would carry it into the output (p480: max error 0.0203
  // of the RMS against the correctly rounded output's 0.0194).  Second pass:
  // q'' = fp16(q^ / 8), exact (a power of two), so a score is the fp32 sum of
  // exact products, q^.k^ / 8 (and m, the bias and the raises are in those
  // units), and each exponential first multiplies by 8 c in fp32 -- one more
  // VALU operation per score, in the pass that only peaked rows take.
  const float q_scale = kRobust ? 0.125f : c_log2;
  const float c_exp = c_log2 * 8.0f;
  auto exp2_score = [&](float x) __attribute__((always_inline)) {
    return __builtin_amdgcn_exp2f(kRobust ? x * c_exp : x);
  };
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int hh = lane >> 5;
  const int l32 = lane & 31;
  int bh, qt;
  if (kSparse) {
    // Slab-synchronous, frame-strided order.  A slab's query tiles are taken
    // in the order of sparse_order_stride (o = 0 .. R S - 1 is tile
    // (o % R) S + o / R, S tiles to a frame: runs of one place in the frame,
    // one tile per frame), and XCD x takes positions [x c, x c + c) of every
    // slab in turn (c = ceil(R S / 8); the grid holds 8 c workgroups per
    // slab).  The workgroups an XCD runs side by side then hold the same
    // patch of different frames, whose kept key blocks -- that patch in every
    // frame -- mostly agree, and walk them in the same order (below), so L2
    // serves most of their copies; the eight XCDs work on about one slab at a
    // time, whose K/V stays in the memory-side cache.  Positions past the
    // slab's tiles leave.
    const int S = sparse_order_stride(g.hw);
    const int c = (sparse_order_len(n_qtiles, S) + kXcds - 1) / kXcds;
    const int x = blockIdx.x % kXcds, l = blockIdx.x / kXcds;
    bh = l / c;
    qt = sparse_order_block(x * c + (l - bh * c), n_qtiles, S);
    if (qt < 0) return;  // the whole workgroup, before any barrier
  } else {
    const int wg = xcd_local_id(blockIdx.x, gridDim.x);
    bh = wg / n_qtiles;
    qt = wg - bh * n_qtiles;
  }
  const int Nq = g.n;  // query rows of the slab (the grid describes them)
  const int N = n_keys;  // keys of the slab
  const size_t slab = (size_t)bh * Nq * D;
  const uint16_t* __restrict__ qs = q + slab;
  const int n_tiles = (N + BN2 - 1) / BN2;
  const size_t pslab = (size_t)bh * n_tiles * kPrepTileElems;
  // Materialise the output pointer now: a kernel-argument load left in flight
  // into the main loop makes every LDS wait there a full lgkmcnt(0).
  uint16_t* out_slab = out + slab;
  asm volatile("" : "+s"(out_slab));
  // out_format 1: one E4M3 byte per element instead of a bf16 pair; 2: one
  // block-INT8 record of kOutRecBytes per row, token-major over `heads`
  const bool out_fp8 = out_format == 1;
  constexpr bool out_rec = kOutRec;
  uint8_t* out8_slab = reinterpret_cast<uint8_t*>(out) + slab;
  asm volatile("" : "+s"(out8_slab), "+s"(out_format));
  const int ob = bh / heads;
  uint8_t* outrec_slab =
      reinterpret_cast<uint8_t*>(out) + ((size_t)ob * Nq * heads + (bh - ob * heads)) * kOutRecBytes;
  const size_t outrec_stride = (size_t)heads * kOutRecBytes;
  const int qrow_first = qt * BM + wave * 64 + l32;
  // Tiles the workgroup walks: every tile of the slab, or the listed blocks'.
  int n_kv = (N + BN2 - 1) / BN2;
  int last_blk = 0, last_pos = 0;  // sparse: the last key block and its walk position
  if (kSparse) {
    // counts and entries are clamped to the slab, whatever the list holds, so
    // every copy stays inside the slab's prepared tiles
    const size_t qb = (size_t)bh * n_qtiles + qt;
    const int cnt = min(max(counts[qb], 1), min(nkb, kMaxSparseBlocks));
    auto listed = [&](int e) { return min((int)blocks[qb * nkb + e], nkb - 1); };
    // Every workgroup walks its ascending list from the first entry: those
    // running side by side, whose lists mostly agree, then fetch the same key
    // blocks at about the same time.  (A full list is the dense walk.)
    const int pos0 = 0;
    auto entry = [&](int e) { return (uint32_t)listed((pos0 + min(e, cnt - 1)) % cnt); };
    for (int e = tid; e < cnt; e += 256) blist[e] = entry(e) | entry(e + 1) << 16;
    n_kv = 4 * cnt;
    // the list's last (largest) block -- the only one that can hold keys past
    // N -- and where the walk meets it
    last_blk = __builtin_amdgcn_readfirstlane(listed(cnt - 1));
    last_pos = __builtin_amdgcn_readfirstlane((cnt - 1 - pos0 + cnt) % cnt);
    __syncthreads();
  }
  // Slab tile of walk position t (clamped to the walk; a listed block's
  // tiles past the slab's last are clamped by the copy and masked whole).
  auto walk_tile = [&](int t) __attribute__((always_inline)) {
    if (!kSparse) return t;
    t = min(t, n_kv - 1);
    return 4 * __builtin_amdgcn_readfirstlane((int)(blist[t >> 2] & 0xFFFFu)) + (t & 3);
  };
  // First key of walk position t where it may need masking: in the sparse
  // walk only the last listed block's tiles can hold keys past N (every other
  // block is whole); elsewhere 0, never masked (N >= 32 whenever a slab has
  // two blocks).
  auto mask_kv0 = [&](int t) __attribute__((always_inline)) {
    if (!kSparse) return t * BN2;
    return (t >> 2) == last_pos ? (4 * last_blk + (t & 3)) * BN2 : 0;
  };
  if (kRobust) {
    // Second pass: only the row blocks the first pass marked (NaN rows) are
    // recomputed; every other workgroup leaves at once.
    bool marked = false;
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
      const int row = qrow_first + 32 * qb;
      if (hh == 0 && row < Nq)
        marked |= out_rec   ? outrec_slab[row * outrec_stride + 128] == 0xFF
                  : out_fp8 ? (out8_slab[(size_t)row * D] & 0x7F) == 0x7F
                            : (out_slab[(size_t)row * D] & 0x7FFF) > 0x7F80;
    }
    if (!__syncthreads_or(marked)) return;
  }

  // ---- Q' fragments of the wave's two 32-row blocks, normalised (q_gamma)
  // and rotated in the load.  A lane holds the even (hh = 0) or odd chunks of
  // its row; the sum of squares pairs them across the lane halves first, then
  // runs the rest of the fixed tree in the lane.
  const int qrow0 = qrow_first;  // block qb holds row qrow0 + 32 qb
  f16x8 qf[2][8];
  bool bad_q = false;  // |q^| log2(e)/sqrt(D) out of fp16's range (or not finite)
#pragma unroll
  for (int qb = 0; qb < 2; ++qb) {
    const int row = min(qrow0 + 32 * qb, Nq - 1);
    Pos p{0, 0, 0, false};
    if (kRope) p = token_pos(row, g);
    uint4 x[8];
    if (kRec) {
      // q decoded from the row's block-INT8 record (token-major, `heads`
      // records per token), already normalised and rotated
      const int b = bh / heads;
      const uint8_t* r = qrec + (((size_t)b * Nq + row) * heads + (bh - b * heads)) * kRecBytes;
#pragma unroll
      for (int kk = 0; kk < 8; ++kk) x[kk] = rec_chunk(r, 0, 2 * kk + hh);
    } else {
      const uint4* src = reinterpret_cast<const uint4*>(qs + (size_t)row * D);
#pragma unroll
      for (int kk = 0; kk < 8; ++kk) x[kk] = src[2 * kk + hh];
    }
    float inv = 1.0f;
    if (q_gamma != nullptr) {
      float s1[8];
#pragma unroll
      for (int kk = 0; kk < 8; ++kk) {
        const float pk = chunk_sumsq(x[kk]);
        s1[kk] = pk + __shfl_xor(pk, 32);  // chunks 2kk and 2kk + 1
      }
      const float s3a = (s1[0] + s1[1]) + (s1[2] + s1[3]);
      const float s3b = (s1[4] + s1[5]) + (s1[6] + s1[7]);
      inv = rms_inv(s3a + s3b, eps);
    }
#pragma unroll
    for (int kk = 0; kk < 8; ++kk) {
      const int cc = 2 * kk + hh;
      // kRope: prefix rows turn by the origin's table entries, an exact identity
      const uint4 y = qk_chunk(x[kk], q_gamma, inv, cc, kRope, tab, tab_lo_plane(tab, g), kRope ? tab_pair(cc, p, g) : 0);
      qf[qb][kk] = bf16x8_to_f16x8_scaled(y, q_scale);
      bad_q |= f16x8_nonfinite(__builtin_bit_cast(uint4, qf[qb][kk]));
    }
  }
  note_range(bad_q, SOL_RANGE_Q);

  // ---- staging: each prepared tile (8 KB) is copied into LDS by buffer loads
  // that write LDS directly: wave w moves the 1 KB blocks 2w and 2w + 1.  Tile
  // indices past the end are clamped (the copies are never read).
  const int wave_s = __builtin_amdgcn_readfirstlane(wave);
  const uint32_t slab_bytes = (uint32_t)n_tiles * (kPrepTileElems * 2);
  const __amdgpu_buffer_rsrc_t rsrc_k =
      __builtin_amdgcn_make_buffer_rsrc((void*)(k + pslab), (short)0, (int)slab_bytes, kBufferDword3);
  const __amdgpu_buffer_rsrc_t rsrc_v =
      __builtin_amdgcn_make_buffer_rsrc((void*)(v + pslab), (short)0, (int)slab_bytes, kBufferDword3);
  // One 1 KB block per call, as inline assembly: through the builtin the
  // compiler would wait for every copy in flight (vmcnt 0) before any read of
  // the same LDS array, since it cannot tell the ring's buffers apart; here
  // dma_barrier() alone orders the copies.  M0 carries the LDS base of the
  // copy, with the one wait state a VMEM read of M0 needs after an SALU write
  // of it.  M0 is declared clobbered: the compiler itself uses M0 nowhere in
  // these kernels (no LDS DMA builtin, no indirect register indexing, no
  // message), which a build test checks on the generated code.
  auto dma_blk = [&](const __amdgpu_buffer_rsrc_t& rs, uint16_t* lds_tile, int tile, int u)
      __attribute__((always_inline)) {
    const uint32_t tb = (uint32_t)min(tile, n_tiles - 1) * (kPrepTileElems * 2);
    const int blk = 2 * wave_s + u;
    const uint32_t lds_addr = (uint32_t)(uintptr_t)(
        (__attribute__((address_space(3))) uint16_t*)(lds_tile + blk * 512));
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"  // M0 is a reserved register
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, %3 offen lds"
                 :
                 : "s"(lds_addr), "v"(lane * 16), "s"(rs), "s"(tb + blk * 1024)
                 : "memory", "m0");
#pragma clang diagnostic pop
  };
  // Walk position t lands in ring slot t; the copy reads slab tile `tile`.
  auto dma_k = [&](int t, int tile, int u) __attribute__((always_inline)) {
    dma_blk(rsrc_k, k_lds + (t & (kKBufs - 1)) * kPrepTileElems, tile, u);
  };
  auto dma_v = [&](int t, int tile, int u) __attribute__((always_inline)) {
    dma_blk(rsrc_v, v_lds + (t & (kVB - 1)) * kPrepTileElems, tile, u);
  };
  // Fragment kk of K tile `tile` / fragment j = 4 kst + db of V tile `tile`.
  auto kfrag = [&](int tile, int kk) __attribute__((always_inline)) {
    return *reinterpret_cast<const f16x8*>(k_lds + (tile & (kKBufs - 1)) * kPrepTileElems + kk * 512 + lane * 8);
  };
  auto vfrag = [&](int tile, int j) __attribute__((always_inline)) {
    return *reinterpret_cast<const f16x8*>(v_lds + (tile & (kVB - 1)) * kPrepTileElems + j * 512 + lane * 8);
  };

  f32x16 o[2][4];
#pragma unroll
  for (int qb = 0; qb < 2; ++qb)
#pragma unroll
    for (int db = 0; db < 4; ++db) o[qb][db] = f32x16{};
  float m_ref[2];   // reference max of each query row (units of c q.k)
  f32x16 bias[2];   // -m_ref, the first addend of every score chain
  float l_run[2] = {0.0f, 0.0f};
  float ovf = 0.0f;  // first pass: largest per-lane tile sum (above 2^15: rows marked)

  // Register j of a score block holds key 8(j/4) + 4hh + (j%4) of the tile;
  // the tile's first key is kv0.
  auto mask_tile = [&](int kv0, f32x16* s) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const int key = kv0 + 8 * (j >> 2) + 4 * hh + (j & 3);
      if (key >= N) {
        s[0][j] = -__builtin_inff();
        s[1][j] = -__builtin_inff();
      }
    }
  };
  auto mask_block = [&](int kv0, f32x16& s) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < 16; ++j)
      if (kv0 + 8 * (j >> 2) + 4 * hh + (j & 3) >= N) s[j] = -__builtin_inff();
  };
  auto tile_max = [&](const f32x16& s) __attribute__((always_inline)) {
    float mx = fmaxf(s[0], s[1]);
#pragma unroll
    for (int j = 2; j < 16; j += 2) mx = fmaxf(fmaxf(mx, s[j]), s[j + 1]);
    return fmaxf(mx, __shfl_xor(mx, 32));
  };
  // Slab tiles of iteration i's copies, K(i + kKAhead) and V(i + kVAhead);
  // pair: the sparse walk's list word of walk position i + kVAhead (and the
  // next entry).
  auto copy_tiles = [&](int i, uint32_t pair, int& tile_k, int& tile_v) __attribute__((always_inline)) {
    tile_k = i + kKAhead;
    tile_v = i + kVAhead;
    if (kSparse) {
      const uint32_t w = __builtin_amdgcn_readfirstlane(pair);
      const int tv = min(i + kVAhead, n_kv - 1), tk = min(i + kKAhead, n_kv - 1);
      const int lo = (int)(w & 0xFFFFu), hi = (int)(w >> 16);
      tile_v = 4 * lo + (tv & 3);
      tile_k = 4 * ((tk >> 2) == (tv >> 2) ? lo : hi) + (tk & 3);
    }
  };
  // Raise the reference max of query block qb to the largest score of tile
  // s (scores held against the current m, keys past N at -inf) where that
  // is larger: O and l are rescaled, s (and s_next, the block's scores of the
  // next tile when they exist) move to the new m, and the tile's fp16 words
  // and their sum are redone.  Exact: numerator and denominator keep one
  // reference.
  auto raise_max = [&](int qb, f32x16& s, f32x16* s_next, uint32_t* words, float& lsum)
      __attribute__((always_inline)) {
    const float delta = fmaxf(tile_max(s), 0.0f);
    const float alpha = exp2_score(-delta);
    m_ref[qb] += delta;
    l_run[qb] *= alpha;
#pragma unroll
    for (int db = 0; db < 4; ++db) o[qb][db] *= alpha;
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      s[j] -= delta;
      if (s_next) (*s_next)[j] -= delta;
      bias[qb][j] -= delta;
    }
    float la = 0.0f, lb = 0.0f;
#pragma unroll
    for (int w = 0; w < 8; ++w) {
      const float ea = exp2_score(s[2 * w]);
      const float eb = exp2_score(s[2 * w + 1]);
      words[w] = pack_f16x2(ea, eb);
      la += ea;
      lb += eb;
    }
    lsum = la + lb;
  };
  // Fragment registers, a whole tile ahead: kr[kk] holds fragment kk of the K
  // tile being multiplied (then of the next one), vr[j] fragment j of the V
  // tile (then of the next one).
  f16x8 kr[8];
  f16x8 vr[8];
  // Words of P(i): qb0 words come from the previous phase B, qb1 words from
  // this phase A.  l0/l1 are their row sums over the tile.
  // Iteration i:
  //   phase A (8 slot pairs): S(i+1) MFMAs (qb0, then qb1, per K fragment) +
  //     P(i) qb1 word j
  //   phase B (8 slot pairs): PV(i) MFMAs (qb0, then qb1, per V fragment) +
  //     P(i+1) qb0 word j; the overflow check of P(i) qb1 between the first
  //     two, that of P(i+1) qb0 at the end
  auto iteration = [&](int i, f32x16* cs, f32x16* ns, uint32_t* p0_cur, uint32_t* p0_next,
                       float& l0_cur, float& l0_next) __attribute__((always_inline)) {
    // K tile t sits in buffer t % 8 from its copy (iteration t - kKAhead, or
    // the prologue) until the copy of tile t + 8 overwrites it, and is read in
    // iteration t-2 (and by the rare path below in iteration t); V
    // tile t sits in buffer t % kVB from its copy (iteration t - kVAhead) until
    // tile t + kVB's, and is read in iteration t-1.  Every overwrite comes at
    // least two barriers after the last wave consumed the reads of the tile
    // it replaces.
    // Sparse walk: the list word of the tiles this iteration copies, read
    // from LDS now and made scalar in phase A.
    uint32_t pair = 0;  // list word of walk position i + kVAhead (and the next entry)
    if (kSparse) pair = blist[min(i + kVAhead, n_kv - 1) >> 2];
    // ---- phase A
    int tile_k = 0, tile_v = 0;
    uint32_t p1[8];
    float l1;
    uint32_t t01 = 0, t23 = 0, t03 = 0, t45 = 0;  // fp16 pair sums of the words
    float pa = 0.0f, pb = 0.0f;  // the previous pair's probabilities
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      // slot 1: S MFMA of block 0; exponential of register 2j; pack of
      // word j-1.
      if (j == 0) {
        mfma_s_first(ns[0], kr[0], qf[0][0], bias[0]);
      } else {
        mfma_s_next(ns[0], kr[j], qf[0][j]);
      }
      __builtin_amdgcn_sched_barrier(0);
      float ea = exp2_score(cs[1][2 * j]);
      keep(ea);
      if (j > 0) {
        p1[j - 1] = pack_f16x2(pa, pb);
        keep(p1[j - 1]);
      }
      // sparse walk: the slab tiles of phase B's copies (scalar work on the
      // list word) in a slot with little VALU work (0.7 % faster there; the
      // dense walk's trivial tiles stay at phase B's start, where moving
      // them cost it 2 %)
      if (kSparse && j == 3) copy_tiles(i, pair, tile_k, tile_v);
      __builtin_amdgcn_sched_barrier(0);
      // slot 2: S MFMA of block 1; fragment kk = j of K(i+2) into the register
      // just used; exponential of register 2j + 1; a step of the word-sum tree.
      if (j == 0) {
        mfma_s_first(ns[1], kr[0], qf[1][0], bias[1]);
      } else {
        mfma_s_next(ns[1], kr[j], qf[1][j]);
      }
      __builtin_amdgcn_sched_barrier(0);
      // First pass: the iteration's barrier, once its first two score MFMAs
      // (register operands only) are on the matrix cores, which then keep
      // working through the wait; every LDS read and copy of the iteration
      // comes after it.
      if (!kRobust && j == 0) dma_barrier<kInflight>();
      kr[j] = kfrag(i + 2, j);
      if (j == 2) { t01 = add_f16x2(p1[0], p1[1]); keep(t01); }
      if (j == 4) { t23 = add_f16x2(p1[2], p1[3]); keep(t23); }
      if (j == 5) { t03 = add_f16x2(t01, t23); keep(t03); }
      if (j == 6) { t45 = add_f16x2(p1[4], p1[5]); keep(t45); }
      float eb = exp2_score(cs[1][2 * j + 1]);
      keep(eb);
      __builtin_amdgcn_sched_barrier(0);
      pa = ea;
      pb = eb;
    }
    p1[7] = pack_f16x2(pa, pb);
    l1 = sum_f16x2(add_f16x2(t03, add_f16x2(t45, add_f16x2(p1[6], p1[7]))));
    if (kRobust) {
      // Rare: a score of block 1's tile exceeds m by more than 15, so its
      // fp16 words (or their sums) overflowed: raise m while S(i) is still in
      // registers (S(i+1) of the block, computed against the old m, moves
      // with it).
      if (__builtin_expect(__any(l1 > kP16SumLimit), 0)) {
        mfma_wait();  // the inline score MFMAs of S(i+1) have landed
        raise_max(1, cs[1], &ns[1], p1, l1);
      }
    } else {
      ovf = fmaxf(ovf, fmaxf(l0_cur, l1));
    }
    l_run[0] += l0_cur;
    l_run[1] += l1;
    keep(l_run[0]);
    keep(l_run[1]);
    if (!kRobust) keep(ovf);
    // The tail above runs in the shadow of the last score MFMAs and counts
    // toward their latency (pinned here: the compiler would otherwise sink it
    // past the branch below).
    __builtin_amdgcn_sched_barrier(0);
    f16x8 pf[2][2];
    auto words_to_operands = [&](int qb, const uint32_t* w) __attribute__((always_inline)) {
#pragma unroll
      for (int kst = 0; kst < 2; ++kst)
        pf[qb][kst] = __builtin_bit_cast(f16x8, make_uint4(w[4 * kst], w[4 * kst + 1], w[4 * kst + 2],
                                                           w[4 * kst + 3]));
    };
    words_to_operands(0, p0_cur);
    words_to_operands(1, p1);
    // S(i+1) is read by the VALU from here on: its MFMAs must have landed (the
    // tail above and these wait states make the 12 an 8-pass result needs; a
    // build test checks the count), and a ragged last tile is masked first.
    // The empty statement keeps the score MFMAs' results and srcC live up to
    // here: where they are dead (the last iteration) the compiler would
    // otherwise reuse their registers while the MFMAs, invisible to it, still
    // write or read them.
    mfma_wait_tail();
    asm volatile("" ::"v"(ns[0]), "v"(ns[1]), "v"(bias[0]), "v"(bias[1]));
    const int kv_next = mask_kv0(i + 1);  // first key of walk tile i + 1
    if (__builtin_expect(i + 1 < n_kv && kv_next + BN2 > N, 0)) {
      mfma_wait();
      mask_tile(kv_next, ns);
    }
    __builtin_amdgcn_sched_barrier(0);
    // ---- phase B
    pa = pb = 0.0f;
    t01 = t23 = t03 = t45 = 0;
    if (!kSparse) copy_tiles(i, pair, tile_k, tile_v);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int kst = j >> 2, db = j & 3;
      // slot 1: PV MFMA of block 0; exponential of register 2j of S(i+1)
      // block 0; pack of word j-1; a copy block in pairs 1, 2, 3 and 5.
      o[0][db] = __builtin_amdgcn_mfma_f32_32x32x16_f16(vr[j], pf[0][kst], o[0][db], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
      float ea = exp2_score(ns[0][2 * j]);
      keep(ea);
      if (j > 0) {
        p0_next[j - 1] = pack_f16x2(pa, pb);
        keep(p0_next[j - 1]);
      }
      // over K(i + kKAhead - 8), read in iteration i + kKAhead - 10 at the
      // latest (i - 6 in the dense walk, i - 4 in the sparse one); over
      // V(i + kVAhead - kVB), whose fragments every wave read two barriers ago
      if (j == 1) dma_k(i + kKAhead, tile_k, 0);
      if (j == 2) dma_v(i + kVAhead, tile_v, 0);
      if (j == 3) dma_k(i + kKAhead, tile_k, 1);
      if (j == 5) dma_v(i + kVAhead, tile_v, 1);
      __builtin_amdgcn_sched_barrier(0);
      // slot 2: PV MFMA of block 1; fragment j of V(i+1) into the register
      // just used; exponential of register 2j + 1; a step of the word-sum tree.
      o[1][db] = __builtin_amdgcn_mfma_f32_32x32x16_f16(vr[j], pf[1][kst], o[1][db], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
      vr[j] = vfrag(i + 1, j);
      if (j == 2) { t01 = add_f16x2(p0_next[0], p0_next[1]); keep(t01); }
      if (j == 4) { t23 = add_f16x2(p0_next[2], p0_next[3]); keep(t23); }
      if (j == 5) { t03 = add_f16x2(t01, t23); keep(t03); }
      if (j == 6) { t45 = add_f16x2(p0_next[4], p0_next[5]); keep(t45); }
      float eb = exp2_score(ns[0][2 * j + 1]);
      keep(eb);
      __builtin_amdgcn_sched_barrier(0);
      pa = ea;
      pb = eb;
    }
    p0_next[7] = pack_f16x2(pa, pb);
    l0_next = sum_f16x2(add_f16x2(t03, add_f16x2(t45, add_f16x2(p0_next[6], p0_next[7]))));
    keep(p0_next[7]);
    // Second pass: block 0's words of P(i+1) are compared here and branched
    // on after the barrier (not after the last tile: S(n_kv) is a re-read of
    // a real tile, unmasked, whose words are never used).
    uint64_t ovf0 = 0;
    if (kRobust && i + 1 < n_kv) {
      ovf0 = __ballot(l0_next > kP16SumLimit);
      asm volatile("" : "+s"(ovf0));
    }
    // The copies the next iteration reads must have landed: those issued
    // kKAhead - 2 iterations ago (K) and kVAhead - 1 ago (V) -- so only the
    // copies of this and the kInflight - 1 previous iterations (4 each) may
    // still be in flight.  (First pass: that barrier is the next iteration's,
    // after its first two MFMAs.)
    if (kRobust) dma_barrier<kInflight>();
    // Raise block 0's m while S(i+1) is still in registers (the block's next
    // scores are computed with the raised m).
    if (kRobust && __builtin_expect(ovf0 != 0, 0)) raise_max(0, ns[0], nullptr, p0_next, l0_next);
    keep(l0_next);
  };

  // ---- prologue: K(0 .. kKAhead - 2) and V(0 .. kVAhead - 2) in LDS,
  // K(kKAhead - 1) and V(kVAhead - 1) on their way; S(0) against m = its own
  // max; the qb0 words of P(0); the fragment registers loaded with K(1) and
  // V(0).
#pragma unroll
  for (int t = 0; t < kKAhead - 1; ++t) {
    const int wt = walk_tile(t);
    dma_k(t, wt, 0);
    dma_k(t, wt, 1);
    if (t < kVAhead - 1) {
      dma_v(t, wt, 0);
      dma_v(t, wt, 1);
    }
  }
  if (!kRobust && tid == 0) n_gave_up = 0;
  __builtin_amdgcn_s_waitcnt(0x0070);  // vmcnt 0, lgkmcnt 0: every copy so far has landed
  __syncthreads();
  {
    const int wk = walk_tile(kKAhead - 1), wv = walk_tile(kVAhead - 1);
    dma_k(kKAhead - 1, wk, 0);
    dma_k(kKAhead - 1, wk, 1);
    dma_v(kVAhead - 1, wv, 0);
    dma_v(kVAhead - 1, wv, 1);
  }
  // S(0) with the builtin MFMA: outside the hot loop the compiler may stage
  // Q' through temporary AGPRs, and only MFMAs it can see are safe next to
  // such copies.
  f32x16 sa[2], sb[2];
  sa[0] = f32x16{};
  sa[1] = f32x16{};
#pragma unroll
  for (int kk = 0; kk < 8; ++kk) {
    const f16x8 kf = kfrag(0, kk);
    sa[0] = __builtin_amdgcn_mfma_f32_32x32x16_f16(kf, qf[0][kk], sa[0], 0, 0, 0);
    sa[1] = __builtin_amdgcn_mfma_f32_32x32x16_f16(kf, qf[1][kk], sa[1], 0, 0, 0);
  }
  if (mask_kv0(0) + BN2 > N) mask_tile(mask_kv0(0), sa);
  // The reference max also covers each 32-row block's "diagonal" tile -- the
  // keys at the rows' own positions (offset by n_keys - Nq, the layout of a
  // cached prefix of keys) -- where a video DiT's local attention peaks: with
  // the first tile alone, rows whose scores climb 11 or more binades above it
  // would overflow the fp16 word sums and take the rare path again and again.
  // The tile must be one the walk attends (always in the dense walk; looked
  // up in the list for the sparse one), so the reference never exceeds the
  // attended maximum.  Fragments are read straight from the prepared tile in
  // global memory.
  float m_diag[2] = {-__builtin_inff(), -__builtin_inff()};
  {
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
      const int key = min(max(qt * BM + wave * 64 + 32 * qb + (N - Nq), 0), N - 1);
      const int tile = key / BN2;
      bool attended = true;
      if (kSparse) {
        const int blk = key / kSparseKeyBlock;
        bool hit = false;
        for (int e = lane; e < n_kv / 4; e += 64) hit |= (int)(blist[e] & 0xFFFFu) == blk;
        attended = __any(hit);
      }
      if (attended) {
        const f16x8* kg = reinterpret_cast<const f16x8*>(k + pslab + (size_t)tile * kPrepTileElems);
        f32x16 sd = f32x16{};
#pragma unroll
        for (int kk = 0; kk < 8; ++kk)
          sd = __builtin_amdgcn_mfma_f32_32x32x16_f16(kg[kk * 64 + lane], qf[qb][kk], sd, 0, 0, 0);
        if (tile * BN2 + BN2 > N) mask_block(tile * BN2, sd);
        m_diag[qb] = tile_max(sd);
      }
    }
  }
#pragma unroll
  for (int qb = 0; qb < 2; ++qb) {
    // finite: the walk's first tile always holds a valid key
    m_ref[qb] = fmaxf(tile_max(sa[qb]), m_diag[qb]);
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      sa[qb][j] -= m_ref[qb];
      bias[qb][j] = -m_ref[qb];
    }
  }
  uint32_t pA[8], pB[8];
  float lA = 0.0f, lB = 0.0f;
  {
    float la = 0.0f, lb = 0.0f;
#pragma unroll
    for (int w = 0; w < 8; ++w) {
      const float ea = exp2_score(sa[0][2 * w]);
      const float eb = exp2_score(sa[0][2 * w + 1]);
      pA[w] = pack_f16x2(ea, eb);
      la += ea;
      lb += eb;
    }
    lA = la + lb;
  }
#pragma unroll
  for (int t = 0; t < 8; ++t) {
    kr[t] = kfrag(1, t);
    vr[t] = vfrag(0, t);
  }
  mfma_wait();

  int i = 0;
  bool gave_up = false;
  for (; i + 1 < n_kv; i += 2) {
    iteration(i, sa, sb, pA, pB, lA, lB);
    iteration(i + 1, sb, sa, pB, pA, lB, lA);
    // First pass: a wave whose probabilities left the fp16 range stops here
    // (its rows are recomputed by the second pass).  Checked once per loop
    // trip, beside the loop's own branch.
    if (!kRobust && __builtin_expect(__any(ovf > kP16SumLimit), 0)) {
      gave_up = true;
      i += 2;
      break;
    }
  }
  if (gave_up) {
    // The other waves still need this wave's share of every tile copy, and
    // the barriers: one per remaining tile, as their loop does -- until every
    // wave of the workgroup has stopped (the count is raised before a barrier
    // and read after it, so all four see the last raise after the same one).
    if (lane == 0) atomicAdd(&n_gave_up, 1);
    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt 0: the raise is done before the barrier
    for (; i < n_kv; ++i) {
      dma_barrier<kInflight>();  // iteration i's barrier, as in the computing waves
      if (__builtin_amdgcn_readfirstlane(n_gave_up) == kWaves2) break;
      const uint32_t pair = kSparse ? blist[min(i + kVAhead, n_kv - 1) >> 2] : 0u;
      int tile_k, tile_v;
      copy_tiles(i, pair, tile_k, tile_v);
      dma_k(i + kKAhead, tile_k, 0);
      dma_v(i + kVAhead, tile_v, 0);
      dma_k(i + kKAhead, tile_k, 1);
      dma_v(i + kVAhead, tile_v, 1);
    }
  } else if (i < n_kv) {
    iteration(i, sa, sb, pA, pB, lA, lB);
  }

  // ---- epilogue: out = O / l; register j of block (qb, db) is dim 32db + 8(j/4) + 4hh + j%4.
  // A first-pass wave whose probabilities left the fp16 range writes its rows
  // as NaN instead (bf16 0x7FC0, E4M3 0x7F, records with scale codes 0xFF):
  // the second pass recomputes exactly those.
  const bool marked = !kRobust && __any(ovf > kP16SumLimit);
#pragma unroll
  for (int qb = 0; qb < 2; ++qb) {
    const int row = qrow0 + 32 * qb;
    const float l_tot = l_run[qb] + __shfl_xor(l_run[qb], 32);
    const float inv = 1.0f / l_tot;
    if (!marked) {
      // an output that is not finite is reported (operands out of fp16's
      // range, inf or NaN inputs; marked rows are the second pass's): an inf
      // or NaN accumulator, or 1/l, makes the lane's sum of them inf or NaN
      float sum = inv;
#pragma unroll
      for (int db = 0; db < 4; ++db)
#pragma unroll
        for (int j = 0; j < 16; ++j) sum += o[qb][db][j];
      note_range(f32_nonfinite(sum) && row < Nq, SOL_RANGE_OUT);
    }
    if (out_rec) {
      // block-INT8 output record: 32 dims per scale; a group's 32 values sit
      // in this lane's 16 registers of block db and its partner lane's (hh ^ 1)
      if (row >= Nq) continue;  // uniform over the lane pair
      uint8_t* dst = outrec_slab + row * outrec_stride;
      if (marked) {
        if (hh == 0) *reinterpret_cast<uint4*>(dst + 128) = make_uint4(0xFFFFFFFFu, 0u, 0u, 0u);
        continue;
      }
      uint32_t scales = 0;
#pragma unroll
      for (int db = 0; db < 4; ++db) {
        float a = 0.0f;
#pragma unroll
        for (int j = 0; j < 16; ++j) a = fmaxf(a, __builtin_fabsf(o[qb][db][j] * inv));
        a = fmaxf(a, __shfl_xor(a, 32));
        const uint32_t sc = ue5m3_scale_for(a);
        const float sv = ue5m3_value(sc);
        scales |= sc << (8 * db);
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
          uint32_t w = 0;
#pragma unroll
          for (int e = 0; e < 4; ++e) w |= int8_code(o[qb][db][4 * g4 + e] * inv, sv) << (8 * e);
          *reinterpret_cast<uint32_t*>(dst + 32 * db + 8 * g4 + 4 * hh) = w;
        }
      }
      if (hh == 0) *reinterpret_cast<uint4*>(dst + 128) = make_uint4(scales, 0u, 0u, 0u);
      continue;
    }
    if (out_fp8) {
      if (row >= Nq) continue;
      uint8_t* dst = out8_slab + (size_t)row * D;
      if (marked) {
#pragma unroll
        for (int c = 0; c < 4; ++c)
          *reinterpret_cast<uint4*>(dst + 64 * hh + 16 * c) = make_uint4(0x7F7F7F7Fu, 0x7F7F7F7Fu, 0x7F7F7F7Fu, 0x7F7F7F7Fu);
        continue;
      }
#pragma unroll
      for (int db = 0; db < 4; ++db) {
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
          uint32_t w = 0;
#pragma unroll
          for (int e = 0; e < 4; ++e) w |= f32_to_e4m3(o[qb][db][4 * g4 + e] * inv) << (8 * e);
          *reinterpret_cast<uint32_t*>(dst + 32 * db + 8 * g4 + 4 * hh) = w;
        }
      }
      continue;
    }
    if (row < Nq && marked) {
      uint16_t* dst = out_slab + (size_t)row * D;
#pragma unroll
      for (int c = 0; c < 8; ++c)
        *reinterpret_cast<uint4*>(dst + 64 * hh + 8 * c) = make_uint4(0x7FC07FC0u, 0x7FC07FC0u, 0x7FC07FC0u, 0x7FC07FC0u);
    } else if (row < Nq) {
      uint16_t* dst = out_slab + (size_t)row * D;
#pragma unroll
      for (int db = 0; db < 4; ++db) {
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
          uint2 w;
          w.x = pack_bf16x2(o[qb][db][4 * g4] * inv, o[qb][db][4 * g4 + 1] * inv);
          w.y = pack_bf16x2(o[qb][db][4 * g4 + 2] * inv, o[qb][db][4 * g4 + 3] * inv);
          *reinterpret_cast<uint2*>(dst + 32 * db + 8 * g4 + 4 * hh) = w;
        }
      }
    }
  }
}

}  // namespace

hipError_t launch_rope3d(const uint16_t* x, uint16_t* y, int64_t rows, const SeqGrid& g,
                         const float2* tab, const float* gamma, float eps, hipStream_t stream) {
  const int64_t per_slab = (int64_t)g.n * kChunks;
  const int64_t bh_count = rows / g.n;
  const unsigned gx = (unsigned)((per_slab + 255) / 256);
  const unsigned gy = (unsigned)(bh_count < 65535 ? bh_count : 65535);
  hipLaunchKernelGGL(rope3d_kernel, dim3(gx, gy), dim3(256), 0, stream,
                     reinterpret_cast<const uint4*>(x), reinterpret_cast<uint4*>(y), bh_count, g,
                     tab, gamma, eps);
  return hipGetLastError();
}

hipError_t launch_attn_fwd(const uint16_t* q, const uint16_t* k, const uint16_t* v,
                           uint16_t* out, int BH, const SeqGrid& g, const float2* tab,
                           hipStream_t stream) {
  const int n_qtiles = (g.n + BM - 1) / BM;
  const float c_log2 = (float)(1.4426950408889634 / 11.313708498984761);  // log2(e)/sqrt(128)
  const dim3 grid((unsigned)((int64_t)n_qtiles * BH));
  const int tab_pairs = g.tab_pairs;
  if (tab == nullptr)
    hipLaunchKernelGGL((attn_fwd_kernel<false, false>), grid, dim3(kThreads), 0, stream, q,
                       k, v, out, g, tab, 0, n_qtiles, c_log2);
  else if (tab_pairs <= kTabLdsPairs)
    hipLaunchKernelGGL((attn_fwd_kernel<true, true>), grid, dim3(kThreads), 0, stream, q,
                       k, v, out, g, tab, tab_pairs, n_qtiles, c_log2);
  else
    hipLaunchKernelGGL((attn_fwd_kernel<true, false>), grid, dim3(kThreads), 0, stream, q,
                       k, v, out, g, tab, tab_pairs, n_qtiles, c_log2);
  return hipGetLastError();
}

hipError_t launch_prepare_kv(const uint16_t* k, const uint16_t* v, uint16_t* k_prep,
                             uint16_t* v_prep, int BH, const SeqGrid& g, const float2* tab,
                             int key0, int n_kv, const float* gamma, float eps,
                             hipStream_t stream) {
  const int tile0 = key0 / kPrepTile;
  const int tile1 = (key0 + g.n - 1) / kPrepTile;  // last tile holding one of these keys
  const dim3 pgrid((unsigned)(tile1 - tile0 + 1), (unsigned)(BH < 65535 ? BH : 65535));
  if (tab != nullptr)
    hipLaunchKernelGGL((prep_kv_kernel<true, false>), pgrid, dim3(256), 0, stream,
                       reinterpret_cast<const uint4*>(k), reinterpret_cast<const uint4*>(v),
                       reinterpret_cast<uint4*>(k_prep), reinterpret_cast<uint4*>(v_prep),
                       (int64_t)BH, g, tab, key0, n_kv, tile0, gamma, eps, nullptr, 1);
  else
    hipLaunchKernelGGL((prep_kv_kernel<false, false>), pgrid, dim3(256), 0, stream,
                       reinterpret_cast<const uint4*>(k), reinterpret_cast<const uint4*>(v),
                       reinterpret_cast<uint4*>(k_prep), reinterpret_cast<uint4*>(v_prep),
                       (int64_t)BH, g, tab, key0, n_kv, tile0, gamma, eps, nullptr, 1);
  return hipGetLastError();
}

hipError_t launch_prepare_kv_records(const uint8_t* rec, uint16_t* k_prep, uint16_t* v_prep,
                                     int B, int H, int N, int key0, int n_kv, hipStream_t stream) {
  const int BH = B * H;
  const SeqGrid g = make_grid(N, 0, 0, 0);
  const int tile0 = key0 / kPrepTile;
  const int tile1 = (key0 + N - 1) / kPrepTile;
  const dim3 pgrid((unsigned)(tile1 - tile0 + 1), (unsigned)(BH < 65535 ? BH : 65535));
  hipLaunchKernelGGL((prep_kv_kernel<false, true>), pgrid, dim3(256), 0, stream, nullptr, nullptr,
                     reinterpret_cast<uint4*>(k_prep), reinterpret_cast<uint4*>(v_prep),
                     (int64_t)BH, g, nullptr, key0, n_kv, tile0, nullptr, 0.0f, rec, H);
  return hipGetLastError();
}

hipError_t launch_attn_fwd_prepared(const uint16_t* q, const uint16_t* k_prep,
                                    const uint16_t* v_prep, void* out_v, int BH,
                                    const SeqGrid& g, int n_kv, const float2* tab,
                                    const float* q_gamma, float eps, int out_format,
                                    const uint16_t* blocks, const int* counts, int nkb,
                                    hipStream_t stream, const uint8_t* qrec, int heads) {
  uint16_t* out = static_cast<uint16_t*>(out_v);
  const int n_qtiles = (g.n + BM - 1) / BM;
  const float c_log2 = (float)(1.4426950408889634 / 11.313708498984761);  // log2(e)/sqrt(128)
  const bool sparse = blocks != nullptr;
  // the block-sparse walk runs in slab-synchronous, frame-strided order: 8 ceil(R S / 8) per slab
  const int64_t per_slab =
      sparse ? (int64_t)kXcds * ((sparse_order_len(n_qtiles, sparse_order_stride(g.hw)) + kXcds - 1) / kXcds)
             : n_qtiles;
  const dim3 grid((unsigned)(per_slab * BH));
  // First pass, then the second over the row blocks whose probabilities left
  // the fp16 range.
  for (int pass = 0; pass < 2; ++pass) {
    // queries from records: no rotation, no normalisation, dense
    const bool orec = out_format == 2;
    const int sel = (qrec != nullptr ? 8 + pass : (tab != nullptr) * 4 + pass * 2 + sparse) + 10 * orec;
#define SOL_LAUNCH_PREPARED(R, P, S, Q, O)                                                      \
  hipLaunchKernelGGL((attn_prepared_kernel<R, P, S, Q, O>), grid, dim3(256), 0, stream, q,       \
                     k_prep, v_prep, out, g, tab, n_qtiles, c_log2, n_kv, q_gamma, eps,          \
                     out_format, blocks, counts, nkb, qrec, heads)
    switch (sel) {
      case 0: SOL_LAUNCH_PREPARED(false, false, false, false, false); break;
      case 1: SOL_LAUNCH_PREPARED(false, false, true, false, false); break;
      case 2: SOL_LAUNCH_PREPARED(false, true, false, false, false); break;
      case 3: SOL_LAUNCH_PREPARED(false, true, true, false, false); break;
      case 4: SOL_LAUNCH_PREPARED(true, false, false, false, false); break;
      case 5: SOL_LAUNCH_PREPARED(true, false, true, false, false); break;
      case 6: SOL_LAUNCH_PREPARED(true, true, false, false, false); break;
      case 7: SOL_LAUNCH_PREPARED(true, true, true, false, false); break;
      case 8: SOL_LAUNCH_PREPARED(false, false, false, true, false); break;
      case 9: SOL_LAUNCH_PREPARED(false, true, false, true, false); break;
      case 10: SOL_LAUNCH_PREPARED(false, false, false, false, true); break;
      case 11: SOL_LAUNCH_PREPARED(false, false, true, false, true); break;
      case 12: SOL_LAUNCH_PREPARED(false, true, false, false, true); break;
      case 13: SOL_LAUNCH_PREPARED(false, true, true, false, true); break;
      case 14: SOL_LAUNCH_PREPARED(true, false, false, false, true); break;
      case 15: SOL_LAUNCH_PREPARED(true, false, true, false, true); break;
      case 16: SOL_LAUNCH_PREPARED(true, true, false, false, true); break;
      case 17: SOL_LAUNCH_PREPARED(true, true, true, false, true); break;
      case 18: SOL_LAUNCH_PREPARED(false, false, false, true, true); break;
      default: SOL_LAUNCH_PREPARED(false, true, false, true, true); break;
    }
#undef SOL_LAUNCH_PREPARED
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

namespace {
std::mutex g_flags_mutex;
void* g_flags_ptr[64];  // per device, resolved on first use
}  // namespace

hipError_t range_status(unsigned* flags, bool clear) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
  void* ptr;
  {
    std::lock_guard<std::mutex> lock(g_flags_mutex);
    if (!g_flags_ptr[dev]) {
      e = hipGetSymbolAddress(&g_flags_ptr[dev], HIP_SYMBOL(range_flags));
      if (e != hipSuccess) return e;
    }
    ptr = g_flags_ptr[dev];
  }
  if ((e = hipDeviceSynchronize()) != hipSuccess) return e;
  if ((e = hipMemcpy(flags, ptr, sizeof(unsigned), hipMemcpyDeviceToHost)) != hipSuccess) return e;
  if (clear) {
    const unsigned zero = 0;
    e = hipMemcpy(ptr, &zero, sizeof(unsigned), hipMemcpyHostToDevice);
  }
  return e;
}

}  // namespace sol
