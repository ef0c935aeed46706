// Block routing of the block-sparse attention (Sec. 3.4, "Per-step dynamic
// sparsity" and "Safety rails and the exact prefix KV sink"), for gfx950.
//
// For the self-attention of each (b, h) slab of N tokens, with query blocks of
// 256 rows (the attention kernel's workgroup tile) and key blocks of 128 keys
// (four prepared tiles), both counted from token 0:
//   qbar_I = mean of q^ over block I's rows   (q^ as the attention kernel's
//            query load makes it: normalised, rotated, rounded to bf16),
//   kbar_J = mean of k^ over block J's keys   (read from the prepared tiles),
//   s_IJ   = <qbar_I, kbar_J> / sqrt(D),
//   mu_I, sigma_I = mean and population standard deviation over all J,
//   J is kept for I iff s_IJ > mu_I + tau sigma_I, or J holds a prefix key
//   (the exact prefix sink), or J is I's first best block (no block attends
//   to nothing); a query block holding a prefix row keeps every J.
// The kept blocks of I are written in ascending order, with their count, for
// the block-sparse attention kernel to walk.
//
// Three launches, all small next to the attention: pool_q_kernel (reads q
// once), pool_k_kernel (reads the prepared K once), route_kernel (four query
// blocks per workgroup: the scores go to LDS, mean and spread are fixed-order
// tree reductions, and the kept blocks are compacted with wave ballots).
#include "sol_device.h"

namespace sol {
namespace {

constexpr int kQB = kSparseQueryBlock;
constexpr int kKB = kSparseKeyBlock;
constexpr int kMaxKeyBlocks = kMaxSparseBlocks;

// Mean of q^ over each query block.  Grid (nqb, slabs); 256 threads = 16 rows
// x 16 chunks per step, 16 steps over the block's rows: each thread sums its
// chunk's 8 entries over its 16 rows in row order, then the 16 row groups are
// summed in LDS in group order.
__global__ __launch_bounds__(256) void pool_q_kernel(const uint4* __restrict__ q,
                                                     float* __restrict__ qbar, int64_t bh_count,
                                                     SeqGrid g, const float2* __restrict__ tab,
                                                     const float* __restrict__ gamma, float eps,
                                                     int nqb) {
  __shared__ float part[16][D + 4];
  lds_poison(&part[0][0], sizeof(part));
  lds_poison_done();
  const int N = g.n;
  const int I = blockIdx.x;
  const int t = threadIdx.x, cc = t & 15, rg = t >> 4;
  const int r0 = I * kQB;
  const int rows = min(kQB, N - r0);
  const uint4 zero = make_uint4(0u, 0u, 0u, 0u);
  for (int64_t bh = blockIdx.y; bh < bh_count; bh += gridDim.y) {
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    for (int step = 0; step < kQB / 16; ++step) {
      const int n = r0 + 16 * step + rg;
      const bool valid = n < N;  // the 16 lanes of a row agree
      const uint4 x = valid ? q[((size_t)bh * N + n) * kChunks + cc] : zero;
      const float inv = gamma ? rms_inv(row_sumsq_lanes16(chunk_sumsq(x)), eps) : 1.0f;
      Pos p{0, 0, 0, false};
      if (tab != nullptr && valid) p = token_pos(n, g);
      const bool rot = tab != nullptr && p.rot;
      const uint4 y = valid ? qk_chunk(x, gamma, inv, cc, rot, tab, tab_lo_plane(tab, g), rot ? tab_pair(cc, p, g) : 0) : zero;
      float f[8];
      unpack_bf16x8(y, f);
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[e] += f[e];
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) part[rg][8 * cc + e] = acc[e];
    __syncthreads();
    if (t < D) {
      float sum = 0.0f;
      for (int r = 0; r < 16; ++r) sum += part[r][t];
      qbar[((size_t)bh * nqb + I) * D + t] = sum / (float)rows;
    }
    __syncthreads();
  }
}

// Mean of k^ over each key block, from the prepared K tiles (fp16 k^, exact;
// keys past N are zero there and add nothing).  Grid (nkb, slabs); thread t
// reads the 16-byte fragment slots t and t + 256 of each of the block's four
// tiles -- always key r = t & 31 of a tile, chunks 2(t >> 6) + hh and that +
// 8, hh = (t >> 5) & 1 -- and the 32 keys of a wave half are summed by a
// butterfly over lane bits 0..4.
__global__ __launch_bounds__(256) void pool_k_kernel(const uint4* __restrict__ kp,
                                                     float* __restrict__ kbar, int64_t bh_count,
                                                     int N, int nkb) {
  const int J = blockIdx.x;
  const int t = threadIdx.x;
  const int n_tiles = (N + kPrepTile - 1) / kPrepTile;
  const int keys = min(kKB, N - J * kKB);
  const int kk = t >> 6, hh = (t >> 5) & 1;
  for (int64_t bh = blockIdx.y; bh < bh_count; bh += gridDim.y) {
    float acc[2][8];
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[u][e] = 0.0f;
    for (int tt = 0; tt < 4; ++tt) {
      const int tile = 4 * J + tt;
      if (tile >= n_tiles) break;  // uniform
      const uint4* src = kp + ((size_t)bh * n_tiles + tile) * (kPrepTileElems / 8);
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const uint4 w = src[t + 256 * u];
        const uint32_t h[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const f16x2 pr = __builtin_bit_cast(f16x2, h[e]);
          acc[u][2 * e] += (float)pr[0];
          acc[u][2 * e + 1] += (float)pr[1];
        }
      }
    }
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        float x = acc[u][e];
        x += __shfl_xor(x, 1);
        x += __shfl_xor(x, 2);
        x += __shfl_xor(x, 4);
        x += __shfl_xor(x, 8);
        x += __shfl_xor(x, 16);
        acc[u][e] = x;
      }
    if ((t & 31) == 0) {
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int dim0 = 16 * (kk + 4 * u) + 8 * hh;
#pragma unroll
        for (int e = 0; e < 8; ++e)
          kbar[((size_t)bh * nkb + J) * D + dim0 + e] = acc[u][e] / (float)keys;
      }
    }
  }
}

// Fixed-order sum over the 256 threads of a workgroup (tree in LDS).
__device__ __forceinline__ float block_sum(float x, float* red) {
  const int t = threadIdx.x;
  red[t] = x;
  __syncthreads();
  for (int s = 128; s > 0; s >>= 1) {
    if (t < s) red[t] = red[t] + red[t + s];
    __syncthreads();
  }
  const float r = red[0];
  __syncthreads();
  return r;
}

// Routing of kRouteQB consecutive query blocks per workgroup (each pooled key
// block read from L2 serves all of them).  Grid (ceil(nqb / kRouteQB),
// slabs).  Scores go to LDS; per query block the mean and the spread are
// fixed-order tree reductions, the best block a (score, lowest index)
// reduction, and the kept blocks are compacted in ascending order with wave
// ballots -- the same arithmetic, in the same order, for every block of a
// workgroup.
constexpr int kRouteQB = 4;

__global__ __launch_bounds__(256) void route_kernel(const float* __restrict__ qbar,
                                                    const float* __restrict__ kbar,
                                                    uint16_t* __restrict__ blocks,
                                                    int* __restrict__ counts, int64_t bh_count,
                                                    int nqb, int nkb, int n_prefix, float tau,
                                                    float scale) {
  __shared__ float qs[kRouteQB][D];
  __shared__ float sc[kRouteQB][kMaxKeyBlocks];
  __shared__ float red[256];
  __shared__ int redi[256];
  __shared__ int wcount[4];
  lds_poison(&qs[0][0], sizeof(qs));
  lds_poison(&sc[0][0], sizeof(sc));
  lds_poison(red, sizeof(red));
  lds_poison_done();
  const int I0 = blockIdx.x * kRouteQB;
  const int nq = min(kRouteQB, nqb - I0);
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  for (int64_t bh = blockIdx.y; bh < bh_count; bh += gridDim.y) {
    for (int e = t; e < kRouteQB * D; e += 256) {
      const int u = e / D, d = e % D;
      qs[u][d] = u < nq ? qbar[((size_t)bh * nqb + I0 + u) * D + d] : 0.0f;
    }
    __syncthreads();
    // scores of every query block, this thread's share of their sums, its
    // first best block
    float psum[kRouteQB], best_v[kRouteQB];
    int best_j[kRouteQB];
#pragma unroll
    for (int u = 0; u < kRouteQB; ++u) {
      psum[u] = 0.0f;
      best_v[u] = -__builtin_inff();
      best_j[u] = nkb;
    }
    for (int J = t; J < nkb; J += 256) {
      const float4* kr = reinterpret_cast<const float4*>(kbar + ((size_t)bh * nkb + J) * D);
      float dot[kRouteQB];
#pragma unroll
      for (int u = 0; u < kRouteQB; ++u) dot[u] = 0.0f;
      for (int d4 = 0; d4 < D / 4; ++d4) {
        const float4 kv = kr[d4];
#pragma unroll
        for (int u = 0; u < kRouteQB; ++u) {
          dot[u] = __builtin_fmaf(qs[u][4 * d4], kv.x, dot[u]);
          dot[u] = __builtin_fmaf(qs[u][4 * d4 + 1], kv.y, dot[u]);
          dot[u] = __builtin_fmaf(qs[u][4 * d4 + 2], kv.z, dot[u]);
          dot[u] = __builtin_fmaf(qs[u][4 * d4 + 3], kv.w, dot[u]);
        }
      }
#pragma unroll
      for (int u = 0; u < kRouteQB; ++u) {
        const float sv = dot[u] * scale;
        sc[u][J] = sv;
        psum[u] += sv;
        if (sv > best_v[u]) {
          best_v[u] = sv;
          best_j[u] = J;
        }
      }
    }
    for (int u = 0; u < nq; ++u) {  // uniform
      const int I = I0 + u;
      const size_t qi = (size_t)bh * nqb + I;
      const bool dense = I * kQB < n_prefix;  // the block holds a prefix row
      const float mu = block_sum(psum[u], red) / (float)nkb;
      float pvar = 0.0f;
      for (int J = t; J < nkb; J += 256) {
        const float d = sc[u][J] - mu;
        pvar = __builtin_fmaf(d, d, pvar);
      }
      const float var = block_sum(pvar, red) / (float)nkb;
      const float thr = mu + tau * __builtin_sqrtf(var);
      // first best block: largest score, lowest index among equals
      red[t] = best_v[u];
      redi[t] = best_j[u];
      __syncthreads();
      for (int s = 128; s > 0; s >>= 1) {
        if (t < s) {
          const float ov = red[t + s];
          const int oi = redi[t + s];
          if (ov > red[t] || (ov == red[t] && oi < redi[t])) {
            red[t] = ov;
            redi[t] = oi;
          }
        }
        __syncthreads();
      }
      const int best = redi[0];
      __syncthreads();
      // kept blocks, compacted in ascending order
      int base = 0;
      uint16_t* out = blocks + qi * nkb;
      for (int c0 = 0; c0 < nkb; c0 += 256) {
        const int J = c0 + t;
        const bool keep = J < nkb && (dense || J * kKB < n_prefix || J == best || sc[u][J] > thr);
        const uint64_t m = __ballot(keep);
        const int before = __popcll(m & ((1ull << lane) - 1ull));
        if (lane == 0) wcount[wave] = __popcll(m);
        __syncthreads();
        int off = base;
        for (int w = 0; w < wave; ++w) off += wcount[w];
        if (keep) out[off + before] = (uint16_t)J;
        base += wcount[0] + wcount[1] + wcount[2] + wcount[3];
        __syncthreads();
      }
      if (t == 0) counts[qi] = base;
    }
  }
}

}  // namespace

hipError_t launch_sparse_route(const uint16_t* q, const uint16_t* k_prep, int BH, const SeqGrid& g,
                               const float2* tab, const float* q_gamma, float eps, float tau,
                               void* workspace, hipStream_t stream) {
  const int N = g.n;
  const int nqb = (N + kQB - 1) / kQB, nkb = (N + kKB - 1) / kKB;
  size_t off[4];
  sparse_workspace_offsets(BH, N, off);
  char* ws = static_cast<char*>(workspace);
  int* counts = reinterpret_cast<int*>(ws + off[0]);
  uint16_t* blocks = reinterpret_cast<uint16_t*>(ws + off[1]);
  float* qbar = reinterpret_cast<float*>(ws + off[2]);
  float* kbar = reinterpret_cast<float*>(ws + off[3]);
  const unsigned gy = (unsigned)(BH < 65535 ? BH : 65535);
  hipLaunchKernelGGL(pool_q_kernel, dim3(nqb, gy), dim3(256), 0, stream,
                     reinterpret_cast<const uint4*>(q), qbar, (int64_t)BH, g, tab, q_gamma, eps, nqb);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(pool_k_kernel, dim3(nkb, gy), dim3(256), 0, stream,
                     reinterpret_cast<const uint4*>(k_prep), kbar, (int64_t)BH, N, nkb);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(route_kernel, dim3((nqb + kRouteQB - 1) / kRouteQB, gy), dim3(256), 0, stream, qbar,
                     kbar, blocks, counts,
                     (int64_t)BH, nqb, nkb, g.nt, tau, (float)(1.0 / 11.313708498984761));
  return hipGetLastError();
}

}  // namespace sol
