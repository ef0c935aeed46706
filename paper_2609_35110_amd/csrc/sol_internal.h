// Internal interface between the C ABI front end (sol_api.cpp) and the HIP
// launchers (sol_kernels.hip).  Arguments reaching these functions have been
// validated already.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "sol.h"

namespace sol {

constexpr int kHeadDim = 128;

// The default rotary split of the head dims across (t, h, w): D/4, 3D/8, 3D/8.
constexpr int kSplitT = kHeadDim / 4, kSplitH = 3 * kHeadDim / 8, kSplitW = 3 * kHeadDim / 8;

// Latent grid, packing and rotary split of one sequence.  Derived on the host.
// The split is counted in 16-byte chunks of 8 head dims: chunks [0, c_t) turn
// with the frame t, [c_t, c_h) with the row h, [c_h, c_w) with the column w,
// and [c_w, D/8) pass through unrotated.
struct SeqGrid {
  int n;        // tokens per sequence N
  int nt;       // prefix (unrotated) tokens: N - T*Hl*Wl
  int T, Hl, Wl;
  int hw;       // Hl * Wl
  float inv_hw; // 1 / (Hl*Wl), for exact-after-correction division
  float inv_wl; // 1 / Wl
  int c_t, c_h, c_w;  // chunk boundaries of the split (dt/8, (dt+dh)/8, (dt+dh+dw)/8)
  int s_t, s_h, s_w;  // table pairs per position of each axis (dt/2, dh/2, dw/2)
  int tab_h;    // first pair of the row-axis section of the table  (T dt/2)
  int tab_w;    // first pair of the column-axis section  (T dt/2 + Hl dh/2)
  int tab_pairs;  // pairs in the whole table
  int id_pair;  // first pair of a position-0 row: angle 0, (cos, sin) = (1, 0)
};

// dt, dh, dw: multiples of 8 (validated by the caller), dt + dh + dw <= D.
SeqGrid make_grid(int N, int T, int Hl, int Wl, int dt = kSplitT, int dh = kSplitH,
                  int dw = kSplitW);

// gamma != nullptr: RMS-normalise every row with these D weights first.
hipError_t launch_rope3d(const uint16_t* x, uint16_t* y, int64_t rows, const SeqGrid& g,
                         const float2* tab, const float* gamma, float eps, hipStream_t stream);

hipError_t launch_attn_fwd(const uint16_t* q, const uint16_t* k, const uint16_t* v,
                           uint16_t* out, int BH, const SeqGrid& g, const float2* tab,
                           hipStream_t stream);

// Prepared path.  Prepared K/V: per (b, h) slab, ceil(n_kv/32) tiles of 32
// keys, 8 KB of K and 8 KB of V each, in the fragment order of the
// prepared-path kernel.  launch_prepare_kv writes the g.n source keys of every
// slab to keys key0 .. key0 + g.n - 1 of such a sequence of n_kv keys (rotated
// with grid g; normalised first when gamma != nullptr), plus the zero padding
// past n_kv when it covers the last tile.
hipError_t launch_prepare_kv(const uint16_t* k, const uint16_t* v, uint16_t* k_prep,
                             uint16_t* v_prep, int BH, const SeqGrid& g, const float2* tab,
                             int key0, int n_kv, const float* gamma, float eps,
                             hipStream_t stream);
// g.n query rows (rotated with grid g, normalised first when q_gamma !=
// nullptr) against n_kv prepared keys; out is bf16, or FP8 E4M3 bytes when
// out_fp8.
// blocks != nullptr: block-sparse, each 256-row query block attends only to
// the counts[...] key blocks of 128 keys listed for it in blocks (nkb entries
// per query block, ascending).
// out_format: 0 bf16, 1 FP8 E4M3 bytes, 2 block-INT8 output records (144
// bytes per row, token-major over `heads`).  qrec != nullptr: the queries
// come from block-INT8 QKV records instead of q (token-major, `heads` records
// per token: already normalised and rotated, so tab and q_gamma are null;
// dense).  heads: H of the B*H = BH slabs.
hipError_t launch_attn_fwd_prepared(const uint16_t* q, const uint16_t* k_prep,
                                    const uint16_t* v_prep, void* out, int BH,
                                    const SeqGrid& g, int n_kv, const float2* tab,
                                    const float* q_gamma, float eps, int out_format,
                                    const uint16_t* blocks, const int* counts, int nkb,
                                    hipStream_t stream, const uint8_t* qrec, int heads);
// Block-INT8 QKV records (sol_records.hip and the prepare pass), records
// [B][N][H][400]: the encoder (q and k normalised with their gammas and
// rotated with grid g first when tab != nullptr), the standalone decoder
// (bf16 [B][H][N][D] out), and the prepare pass reading k and v from records
// into keys key0 .. key0 + N - 1 of a prepared sequence of n_kv keys.
// The encoder reads row (b, h, n) of q, k and v at element offset
// b sb + h sh + n sn (multiples of 8), its D values contiguous.
hipError_t launch_qkv_encode(const uint16_t* q, const uint16_t* k, const uint16_t* v, uint8_t* rec,
                             int B, int H, const SeqGrid& g, const float2* tab,
                             const float* q_gamma, const float* k_gamma, float eps,
                             int64_t sb, int64_t sh, int64_t sn, hipStream_t stream);
hipError_t launch_qkv_decode(const uint8_t* rec, uint16_t* q, uint16_t* k, uint16_t* v, int B, int H,
                             int N, hipStream_t stream);
hipError_t launch_prepare_kv_records(const uint8_t* rec, uint16_t* k_prep, uint16_t* v_prep,
                                     int B, int H, int N, int key0, int n_kv, hipStream_t stream);
// Tile and block sizes the host sizing below shares with the kernels.
// Prepared K/V tiles: 32 keys, 8 KB of fp16 each for K and for V.
constexpr int kPrepTile = 32;                         // keys per prepared tile
constexpr int kPrepTileElems = kPrepTile * kHeadDim;  // 4096 fp16 = 8 KB
// Block-sparse routing granularity and the longest kept-block list a query
// block's workgroup stages in LDS (4 bytes an entry, beside 128 KB of K and V
// rings: 8064 entries keep the kernel inside 160 KB).
constexpr int kSparseKeyBlock = 128;    // keys per routing key block (4 tiles)
constexpr int kSparseQueryBlock = 256;  // query rows per routing query block
constexpr int kMaxSparseBlocks = 8064;  // key blocks per slab: N <= 1,032,192
// Query rows per workgroup of the fused kernel (sol_attn_fwd).
constexpr int kFusedRows = 256;

// The block-sparse walk's order of a slab's query blocks: S query blocks to a
// frame of hw tokens (hw / 256 rounded; 1 for frames under two blocks or
// without a grid), R = ceil(nqb / S) rows of S, and order position o in
// [0, R S) is block (o % R) S + o / R (none past the last block).  Consecutive
// positions hold the same place in consecutive frames, where a video DiT's
// attention keeps the same key blocks (that patch in every frame).
__host__ __device__ inline int sparse_order_stride(int hw) {
  return hw >= 2 * kSparseQueryBlock ? (hw + kSparseQueryBlock / 2) / kSparseQueryBlock : 1;
}
__host__ __device__ inline int sparse_order_len(int nqb, int stride) { return (nqb + stride - 1) / stride * stride; }
// The query block at order position o (o >= 0), or -1 when none.
__host__ __device__ inline int sparse_order_block(int o, int nqb, int stride) {
  const int rows = (nqb + stride - 1) / stride;
  const int b = (o % rows) * stride + o / rows;
  return o < rows * stride && b < nqb ? b : -1;
}

// fp16 elements of one (b, h) slab of prepared K (or V).
inline int64_t prepared_tile_elems(int N) {
  return (int64_t)((N + kPrepTile - 1) / kPrepTile) * kPrepTileElems;
}

// Block-sparse routing (sol_sparse.hip).  Workspace sections, byte offsets
// off[0..3]: counts int32 [BH][nqb], blocks uint16 [BH][nqb][nkb], pooled
// queries fp32 [BH][nqb][D], pooled keys fp32 [BH][nkb][D] (nqb = ceil(N/256),
// nkb = ceil(N/128)); returns the total size.
inline size_t sparse_workspace_offsets(int BH, int N, size_t off[4]) {
  const size_t nqb = (size_t)(N + kSparseQueryBlock - 1) / kSparseQueryBlock;
  const size_t nkb = (size_t)(N + kSparseKeyBlock - 1) / kSparseKeyBlock;
  auto up = [](size_t x) { return (x + 255) & ~(size_t)255; };
  off[0] = 0;                                              // counts: int32 [BH][nqb]
  off[1] = up(off[0] + (size_t)BH * nqb * 4);              // blocks: uint16 [BH][nqb][nkb]
  off[2] = up(off[1] + (size_t)BH * nqb * nkb * 2);        // qbar: fp32 [BH][nqb][D]
  off[3] = up(off[2] + (size_t)BH * nqb * kHeadDim * 4);   // kbar: fp32 [BH][nkb][D]
  return up(off[3] + (size_t)BH * nkb * kHeadDim * 4);
}
// Largest N the block-sparse path takes (its key-block lists live in LDS).
inline int sparse_max_tokens() { return kMaxSparseBlocks * kSparseKeyBlock; }
// Pools q (rotated with grid g, normalised with q_gamma) and the prepared
// keys, then routes every query block with threshold parameter tau.
hipError_t launch_sparse_route(const uint16_t* q, const uint16_t* k_prep, int BH, const SeqGrid& g,
                               const float2* tab, const float* q_gamma, float eps, float tau,
                               void* workspace, hipStream_t stream);

// Dense fp16 MFMA rate probe (sol_probe.hip): `workgroups` of four waves,
// each issuing 16 MFMAs of 32x32x16 per iteration; operands: 8192 fp16
// values (16 KB); out: one float per thread (workgroups * 256).
hipError_t launch_mfma_probe(const uint16_t* operands, float* out, int workgroups, int iters,
                             hipStream_t stream);

// At least the workgroups of any attention launch over BH slabs of N tokens
// (the caller checks it fits a 1D grid).
inline int64_t attn_max_workgroups(int N, int BH) {
  // the block-sparse grid's frame-strided order pads a slab to at most
  // 2 nqb + 7 positions (its stride is at most nqb)
  return (2 * (int64_t)((N + kFusedRows - 1) / kFusedRows) + 8) * BH;
}

// The current device's sticky range status (sol_range_status): waits for all
// work on the device, copies the flags out, and clears them when asked.
hipError_t range_status(unsigned* flags, bool clear);

// Record msg as the calling thread's last error (sol_last_error) and return
// status: the front end's error path, for entry points in other sources.
int set_error(int status, const char* msg);

}  // namespace sol
