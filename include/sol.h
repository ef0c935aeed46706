/*
 * sol.h -- C ABI of libsol.so: fused 3D rotary embedding + softmax attention
 * for the video DiT self-attention, on AMD Instinct MI355X (gfx950).
 *
 * The operation (the attention that dominates a denoising step, Sec. 3.2
 * "Optimized attention collectives"; its cost grows with the square of the
 * token count, Sec. 3.4): for every batch b and head h,
 *
 *     q^ = bf16(R(pos) q),  k^ = bf16(R(pos) k)      (3D rotary embedding)
 *     out = softmax(q^ k^T / sqrt(D)) v               (no mask, bidirectional)
 *
 * R is the rotary embedding of Sec. 3.5 (fusion group 2, "QK normalization
 * with partial RoPE"), extended to three axes: head dims [0, dt) rotate with
 * the latent frame t, [dt, dt+dh) with the latent row h, [dt+dh, dt+dh+dw)
 * with the latent column w, and any dims past dt+dh+dw pass through unrotated
 * (partial RoPE).  The default split is D/4, 3D/8, 3D/8 (32/48/48 at D = 128,
 * every dim rotated); the entry points with dt, dh, dw arguments take any
 * split of non-negative multiples of 8 with dt+dh+dw <= D.  Within an axis
 * chunk of width d, the interleaved pair (2i, 2i+1) is turned by the angle
 * pos * base^(-2i/d).  bf16(R(pos) x) is the nearest-even bf16 of the exact
 * rotation: the kernels turn each pair in fp64 with cos and sin to 48 bits
 * (the table's two planes) and round once, so they differ from the correctly
 * rounded value only where it lies within about 2^-47 |pair| of a rounding
 * midpoint.  (One exception, the fused kernel's key tiles, is documented at
 * sol_attn_fwd.)
 *
 * Sequence packing follows Sec. 3.4 "Safety rails" (prefix before the target
 * video): of the N tokens, the first Nt = N - T*Hl*Wl form an unrotated
 * prefix (text); token n >= Nt is the latent at r = n - Nt in t-major raster
 * order: t = r / (Hl*Wl), h = (r / Wl) mod Hl, w = r mod Wl.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Tensors are bf16, contiguous [B][H][N][D] (row-major, D fastest), base
 *    pointers 16-byte aligned, device memory.  Offsets are 64-bit.
 *  - Only D = 128 is implemented (SOL_ERR_UNSUPPORTED otherwise).
 *  - The caller owns every buffer (tensors and the rotary table) and keeps
 *    them alive until the work on `stream` completes.  The library never
 *    allocates, frees or synchronises, and keeps no state across calls except
 *    a thread-local error message (and the static per-GPU workspace of
 *    sol_attn_fwd_noalloc).
 *  - Arguments are validated on the host before any HIP call; a rejected call
 *    returns a negative status and launches nothing.  Launch failures return
 *    SOL_ERR_HIP.  Work is asynchronous on `stream` (NULL = the null stream);
 *    device-side faults surface at the caller's next synchronisation.
 *  - Every function is thread-safe.
 */
#ifndef SOL_H
#define SOL_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Same type as hipStream_t. */
typedef struct ihipStream_t* sol_stream_t;

enum {
  SOL_OK = 0,
  SOL_ERR_INVALID_ARG = -1, /* null/misaligned pointer, bad size, aliasing */
  SOL_ERR_UNSUPPORTED = -2, /* valid but not implemented (D != 128, huge N) */
  SOL_ERR_HIP = -3          /* the HIP runtime reported an error */
};

/* Output formats of sol_attn_fwd_prepared_ex, sol_attn_fwd_sparse and
 * sol_attn_fwd_records. */
enum {
  SOL_OUT_BF16 = 0,        /* bf16, round to nearest even (every other entry point) */
  SOL_OUT_FP8_E4M3 = 1,    /* FP8 E4M3 bytes with unit scale (see sol_attn_fwd_prepared_ex) */
  SOL_OUT_INT8_RECORDS = 2 /* block-INT8 output records (see sol_attn_fwd_prepared_ex) */
};

/*
 * Range status (sol_range_status): bits the kernels set, per device and
 * sticky until cleared, when an input leaves the range the computation
 * supports or an output is not finite.  The prepared path (sol_prepare_kv*,
 * sol_attn_fwd_prepared*, sol_attn_fwd_ws, sol_attn_fwd_noalloc, the chunks
 * of sol_attn_fwd, the block-sparse and records paths) multiplies in fp16
 * with fp32 accumulation:
 *   SOL_RANGE_Q: a query value q^ log2(e)/sqrt(D) is not finite in fp16
 *     (|q^| >= about 513,000, or an inf/NaN input);
 *   SOL_RANGE_K: a key value k^ (normalised, rotated, bf16) is not finite in
 *     fp16 (|k^| >= 65520, or inf/NaN);
 *   SOL_RANGE_V: a value v is not finite in fp16 (|v| >= 65520, or inf/NaN);
 *   SOL_RANGE_OUT: an output element is inf or NaN (any attention entry
 *     point: the fused kernel also converts v to fp16 for the second
 *     product, so |v| >= 65520 lands here; inf or NaN inputs too).
 * Such a call's outputs are not finite where the bad operand takes part --
 * never a finite wrong value -- and the bits say why.  fp16's subnormal range
 * keeps an absolute resolution of 2^-24: values below 2^-14 in magnitude lose
 * relative precision but raise no bit.
 */
enum { SOL_RANGE_Q = 1, SOL_RANGE_K = 2, SOL_RANGE_V = 4, SOL_RANGE_OUT = 8 };

/* Largest N the kernels accept (token indices stay exact in float32 arithmetic). */
#define SOL_MAX_TOKENS (1 << 23)

/*
 * Number of floats in the rotary table for head dim D, latent grid
 * T x Hl x Wl and split dt/dh/dw: 4 * (T*dt/2 + Hl*dh/2 + Wl*dw/2).  Returns 0
 * for invalid arguments (D not a positive multiple of 16, a negative extent,
 * a split that is not three non-negative multiples of 8 summing to at most
 * D).  sol_rope3d_table_floats is the default split D/4, 3D/8, 3D/8.
 */
size_t sol_rope3d_table_floats_ex(int D, int T, int Hl, int Wl, int dt, int dh, int dw);
size_t sol_rope3d_table_floats(int D, int T, int Hl, int Wl);

/*
 * Fill a HOST buffer with the rotary table (caller copies it to the device).
 * Two planes of n/2 floats each, n = sol_rope3d_table_floats_ex(D, T, Hl,
 * Wl, dt, dh, dw).  Plane 0 (hi) holds float pairs (cos, sin), computed in
 * double and rounded to float:
 *   [T  rows x dt/2 pairs]  frame axis:  angle t * base^(-2i/dt)
 *   [Hl rows x dh/2 pairs]  row axis:    angle h * base^(-2i/dh)
 *   [Wl rows x dw/2 pairs]  column axis: angle w * base^(-2i/dw)
 * (an axis of width 0 has no section); plane 1 (lo), in the same order, holds
 * what that rounding lost, float(c - hi) for each double c, so that hi + lo
 * carries c to 48 bits.  host_tab must hold n_floats >= n floats; every entry
 * point reads exactly n (the lo plane starts n/2 floats in).  base > 1
 * (10000 for the workloads here).  Host-only: no HIP call.  A device copy is
 * valid only for calls with the same grid and split.  sol_rope3d_table is the
 * default split D/4, 3D/8, 3D/8: the table of every entry point without
 * dt, dh, dw arguments.
 */
int sol_rope3d_table_ex(float* host_tab, size_t n_floats, int D, int T, int Hl, int Wl, int dt,
                        int dh, int dw, double base);
int sol_rope3d_table(float* host_tab, size_t n_floats, int D, int T, int Hl, int Wl, double base);

/*
 * y = bf16(R(pos) x) for every token (prefix tokens copied unchanged).
 * The same bits as the rotation of queries in every attention entry point and
 * of keys in sol_prepare_kv, sol_sparse_route and the record encoder.
 * x, y: [B][H][N][D] bf16; y == x (in place) is allowed, any other overlap
 * is rejected.  0 <= T*Hl*Wl <= N.  rope_tab_dev: device copy of
 * sol_rope3d_table(D, T, Hl, Wl), 16-byte aligned; it may be NULL only when
 * the grid is empty (then every token is prefix and y = x).
 */
int sol_rope3d(const void* x, void* y, int B, int H, int N, int D, int T, int Hl, int Wl,
               const float* rope_tab_dev, sol_stream_t stream);

/*
 * QK normalization ahead of the rotation (Sec. 3.5, fusion group 2, "QK
 * normalization with partial RoPE"), standalone, under the split dt/dh/dw
 * (dims past dt+dh+dw are normalised, not rotated):
 *   y = bf16(R(pos) (x * gamma / sqrt(mean_d(x_d^2) + eps)))
 * per token and head: the root mean square is taken over the head's D entries
 * of the bf16 input (the rounding point the paper keeps ahead of QK
 * normalization, Sec. 3.5 "LoRA fusion"), everything is fp32, and the result
 * is rounded to bf16 once, after the rotation.  Every token is normalised;
 * prefix tokens are not rotated.  gamma_dev: D fp32 weights in device memory,
 * 16-byte aligned, or NULL (no normalisation: exactly sol_rope3d).  eps >= 0
 * and finite (an all-zero row with eps = 0 gives NaN, as the formula does).
 * rope_tab_dev: the table of this grid and split (NULL only when nothing
 * rotates: an empty grid or dt+dh+dw = 0).  Other arguments as sol_rope3d;
 * sol_rope3d is this call with the default split and no normalisation.  The
 * same normalisation runs in the
 * prepared path below (sol_prepare_kv_ex, sol_attn_fwd_prepared_ex), to the
 * same bits: the sum of squares follows one fixed order in every kernel.
 */
int sol_qknorm_rope3d(const void* x, void* y, int B, int H, int N, int D, int T, int Hl, int Wl,
                      int dt, int dh, int dw, const float* rope_tab_dev, const float* gamma_dev,
                      float eps, sol_stream_t stream);

/*
 * out = softmax(q^ k^T / sqrt(D)) v for every (b, h) slab, q^ and k^ rotated
 * and rounded to bf16 as sol_rope3d (exact rotation).  The call allocates
 * nothing and takes no workspace, so it uses the slabs of `out` it has not
 * written yet as one: it walks the slabs front to back in chunks, and for a
 * chunk of c slabs prepares their K and V (sol_prepare_kv, 2 c slabs' worth of
 * fp16 tiles) in the out slabs after the chunk, then attends to them
 * (sol_attn_fwd_prepared), writing the chunk's own out slabs; each chunk is as
 * large as the room after it allows, and of these chunks the call keeps the
 * leading ones that a launch-round model says pay (a chunk too small to fill
 * the chip costs more than running its slabs in the fused kernel).  The
 * slabs after the kept chunks (sol_attn_fwd_plan tells how many slabs the
 * chunks cover: 36 of 40 at 720p, none at the low resolution's 24 x 12,480)
 * run the fused kernel instead, which rotates q and k in its tile
 * loads -- q^ as sol_rope3d, bit for bit; k^, rotated again in every query
 * tile's pass over the keys, in fp32 with the table's hi plane only, within
 * one bf16 ulp of sol_rope3d's and equal to it except where the exact
 * rotation lies within a few 2^-24 |pair| of a rounding midpoint (about 1
 * element in 10^4) -- with bf16 score operands.  Either way: fp32 softmax
 * statistics and accumulators, probabilities rounded to fp16 and v converted
 * to fp16 for the second product, the output rounded to bf16 (nearest even);
 * the chunks take the prepared path's operand ranges and status bits (below),
 * the fused kernel needs |v| < 65504 (else SOL_RANGE_OUT).  A slab's result
 * depends only on its data and on which of the two it ran through.
 * q, k, v, out: [B][H][N][D] bf16, 16-byte aligned; out must not overlap
 * q, k or v (its contents on entry are ignored).  0 <= T*Hl*Wl <= N.
 * rope_tab_dev = NULL or T*Hl*Wl = 0 means plain attention (nothing rotated);
 * otherwise it is the device copy of sol_rope3d_table(D, T, Hl, Wl), 16-byte
 * aligned.
 */
int sol_attn_fwd(const void* q, const void* k, const void* v, void* out, int B, int H, int N,
                 int D, int T, int Hl, int Wl, const float* rope_tab_dev, sol_stream_t stream);

/*
 * The number of leading (b, h) slabs, in [b][h] order, that sol_attn_fwd
 * computes through the prepared path in place for this shape; the remaining
 * B*H minus that run the fused kernel.  Host-only; negative status for
 * invalid shapes.
 */
int sol_attn_fwd_plan(int B, int H, int N, int D);

/*
 * The attention in two stages, for callers that keep prepared K/V (the
 * paper's reference-KV cache, Sec. 5, reuses one key/value set across
 * denoising steps) or that time the stages apart.
 *
 * sol_prepare_kv: one pass over k and v into the prepared-path format.  Per
 * (b, h) slab, ceil(N/32) tiles of 32 keys; each tile is 8 KB of K and 8 KB of
 * V (fp16) in the order the attention kernel's MFMA fragments read them, so a
 * tile is copied into LDS whole and every fragment read is linear:
 *   K tile, 64-lane block kk (0..7), lane l + 32h: K^[key l][dims 16kk+8h..+7],
 *     K^ = fp16(bf16(R(pos) k)) -- the rotation and rounding of sol_rope3d;
 *   V tile, block j = 4s + c (0..7), lane l + 32h, element i (0..7):
 *     fp16(v)[key 16s + 8(i/4) + 4h + i%4][dim 32c + l].
 * Keys past N are zero.  The fp16 conversions are exact for 2^-14 <= |x| <
 * 65504; smaller values keep fp16's 2^-24 absolute resolution, larger ones
 * overflow to inf and raise SOL_RANGE_K / SOL_RANGE_V (sol_range_status).  k_prep, v_prep: device
 * buffers of sol_prepared_kv_bytes(B, H, N, D) bytes each, 16-byte aligned,
 * not overlapping each other, k or v.  rope_tab_dev as in sol_attn_fwd.
 *
 * sol_attn_fwd_prepared: attention on prepared K/V; q is rotated and rounded
 * to bf16 in its tile load, then scaled by log2(e)/sqrt(D) and rounded to
 * fp16 so the score product runs in fp16 with the softmax scale folded in
 * (|q^| log2(e)/sqrt(D) must stay below 65504, else SOL_RANGE_Q).  Two
 * launches on the stream: the first treats every query row with a reference
 * max taken from the first key tile and the rows' diagonal tile, and stops a
 * row block whose probabilities would leave the fp16 range (scores more than
 * 15 binades above that reference), writing it as NaN; the second recomputes
 * exactly those row blocks, raising the reference in place as it goes (any
 * score distribution: p480's 1 % of keys x8 runs at the rate of the dense
 * shapes).  out must not overlap q, k_prep or v_prep.
 *
 * The result differs from the fused kernel's by rounding only (same contract and
 * error bound; the fp16 score operands and the reference max change the last
 * bits).
 */
size_t sol_prepared_kv_bytes(int B, int H, int N, int D);
int sol_prepare_kv(const void* k, const void* v, void* k_prep, void* v_prep, int B, int H, int N,
                   int D, int T, int Hl, int Wl, const float* rope_tab_dev, sol_stream_t stream);
int sol_attn_fwd_prepared(const void* q, const void* k_prep, const void* v_prep, void* out, int B,
                          int H, int N, int D, int T, int Hl, int Wl, const float* rope_tab_dev,
                          sol_stream_t stream);

/*
 * The prepared path, generalised.
 *
 * sol_prepare_kv_ex: the N keys and values of every (b, h) slab of k, v
 * ([B][H][N][D] bf16) become keys key0 .. key0 + N - 1 of a prepared sequence
 * of n_kv keys (buffers of sol_prepared_kv_bytes(B, H, n_kv, D) bytes, the
 * layout of sol_prepare_kv).  The rotation uses this call's own grid T x Hl x
 * Wl and split dt/dh/dw (its first N - T*Hl*Wl keys are an unrotated prefix;
 * rope_tab_dev the table of that grid and split); with k_gamma_dev the keys
 * are RMS-normalised first, as in sol_qknorm_rope3d.  Several calls
 * fill one prepared sequence from several sources -- the paper's reference-KV
 * cache (Sec. 5, "Reference KV caching mechanism"): the reference tokens'
 * keys and values are prepared once, at the first denoising step, and later
 * steps prepare only their own tokens into the rest of the sequence.  Calls
 * write only their own keys (a tile shared with another call's keys is
 * written element by element) and the zero padding past n_kv, so their order
 * does not matter.  0 <= key0, key0 + N <= n_kv <= SOL_MAX_TOKENS.
 * sol_prepare_kv(...) is sol_prepare_kv_ex with key0 = 0, n_kv = N, the
 * default split and no normalisation.
 *
 * sol_attn_fwd_prepared_ex: N query rows per slab (q, out: [B][H][N][D],
 * rotated with the grid T x Hl x Wl and split dt/dh/dw, RMS-normalised first
 * with q_gamma_dev)
 * against the n_kv prepared keys: out = softmax(q^ k^T / sqrt(D)) v over all
 * of them (n_kv may differ from N).  Every key must have been written by a
 * sol_prepare_kv_ex call.  out_format SOL_OUT_BF16: out is bf16 (2 bytes per
 * element); SOL_OUT_FP8_E4M3: out holds one FP8 E4M3 byte per element (OCP
 * E4M3FN: bias 7, 3 mantissa bits, no infinities, 0x7F NaN) with unit scale --
 * the raw E4M3 values the paper's attention hands to the quantized output
 * projection (Sec. 3.3, "Joint optimization with quantized communication") --
 * rounded to nearest even from the fp32 result and saturated at +-448.
 * SOL_OUT_INT8_RECORDS: the paper's block-INT8 output wire format (Sec. 3.2,
 * "Quantized communication"), one record of SOL_OUT_RECORD_BYTES = 144 bytes
 * per row, token-major like the QKV records (row (b, h, n) at byte
 * ((b N + n) H + h) * 144): bytes 0..127 the int8 codes of the 128 output
 * dims, 128..131 the UE5M3 scale codes of dims [32g, 32g + 32), 132..143
 * zero; scales and codes follow the QKV records' rule (sol_qkv_encode),
 * applied to the fp32 result.
 * sol_attn_fwd_prepared(...) is this call with n_kv = N, the default split,
 * no normalisation and bf16 output.
 *
 * gamma pointers: D fp32 device weights, 16-byte aligned, or NULL; eps as in
 * sol_qknorm_rope3d (ignored when the pointer is NULL).  Other arguments,
 * ownership and errors as sol_prepare_kv / sol_attn_fwd_prepared.
 */
int sol_prepare_kv_ex(const void* k, const void* v, void* k_prep, void* v_prep, int B, int H,
                      int N, int key0, int n_kv, int D, int T, int Hl, int Wl, int dt, int dh,
                      int dw, const float* rope_tab_dev, const float* k_gamma_dev, float eps,
                      sol_stream_t stream);
int sol_attn_fwd_prepared_ex(const void* q, const void* k_prep, const void* v_prep, void* out,
                             int B, int H, int N, int n_kv, int D, int T, int Hl, int Wl, int dt,
                             int dh, int dw, const float* rope_tab_dev, const float* q_gamma_dev,
                             float eps, int out_format, sol_stream_t stream);

/*
 * Block-sparse attention (Sec. 3.4, "Per-step dynamic sparsity" and "Safety
 * rails and the exact prefix KV sink"): the paper's training-free routing by
 * online thresholding, for the self-attention of N tokens on prepared K/V.
 *
 * Query blocks of 256 rows and key blocks of 128 keys, both counted from token
 * 0.  With q^, k^ the rows as they enter the products (normalised with
 * q_gamma_dev / the keys' own preparation, rotated, rounded to bf16):
 *   qbar_I = mean of q^ over block I, kbar_J = mean of k^ over block J,
 *   s_IJ = <qbar_I, kbar_J> / sqrt(D)  (fp32; the block-level score),
 *   mu_I, sigma_I = mean and population standard deviation over all J;
 *   key block J is kept for query block I iff s_IJ > mu_I + tau sigma_I, or
 *   J holds a prefix key (the first N - T*Hl*Wl tokens: an exact sink), or J
 *   is I's first largest-score block; a query block holding a prefix row
 *   keeps every key block (prefix queries attend densely).
 * Each query row then attends, exactly, to the keys of its block's kept key
 * blocks only.  tau -> -inf keeps everything (dense); the paper's refinement
 * steps use tau = 1.0, 1.25, 1.5.
 *
 * sol_sparse_route: pools q and the prepared keys (k_prep from
 * sol_prepare_kv[_ex], key0 = 0, n_kv = N) and writes the routing into the
 * workspace: bytes [0, 4*B*H*nqb): int32 counts[b*H + h][I] of kept blocks;
 * from offset ceil256(4*B*H*nqb): uint16 blocks[b*H + h][I][0..nkb), the
 * kept block indices of (b, h, I) in ascending order (the first counts[..]
 * entries are meaningful); then pooled queries and keys (fp32).
 * nqb = ceil(N/256), nkb = ceil(N/128).  tau finite.
 * sol_attn_fwd_sparse: the attention under that routing (the workspace as
 * sol_sparse_route left it), in any output format of sol_attn_fwd_prepared_ex.
 * The workspace is sol_sparse_workspace_bytes(B, H, N, D) bytes of device
 * memory, 16-byte aligned, not overlapping q, k_prep, v_prep or out.
 * N <= 1,032,192 = 8064 key blocks (SOL_ERR_UNSUPPORTED beyond: the
 * kept-block list of a query block is staged in LDS).  Other arguments and errors as sol_attn_fwd_prepared_ex;
 * sol_sparse_workspace_bytes returns 0 for invalid or unsupported sizes.
 */
size_t sol_sparse_workspace_bytes(int B, int H, int N, int D);
int sol_sparse_route(const void* q, const void* k_prep, int B, int H, int N, int D, int T, int Hl,
                     int Wl, int dt, int dh, int dw, const float* rope_tab_dev,
                     const float* q_gamma_dev, float eps, float tau, void* workspace,
                     size_t workspace_bytes, sol_stream_t stream);
int sol_attn_fwd_sparse(const void* q, const void* k_prep, const void* v_prep, void* out, int B,
                        int H, int N, int D, int T, int Hl, int Wl, int dt, int dh, int dw,
                        const float* rope_tab_dev, const float* q_gamma_dev, float eps,
                        const void* workspace, size_t workspace_bytes, int out_format,
                        sol_stream_t stream);

/*
 * Bytes of device workspace sol_attn_fwd_ws needs: room for k_prep then
 * v_prep, 2 * sol_prepared_kv_bytes(B, H, N, D).  0 for invalid sizes.
 */
size_t sol_attn_workspace_bytes(int B, int H, int N, int D);

/*
 * sol_prepare_kv into the caller's workspace, then sol_attn_fwd_prepared:
 * the rotation of K done once per token instead of once per query tile.
 * Same result as those two calls, bit for bit.  workspace: device memory of at
 * least sol_attn_workspace_bytes(B, H, N, D) bytes, 16-byte aligned, not
 * overlapping q, k, v or out; its contents on entry are ignored and on exit
 * hold k_prep then v_prep.  Other arguments and errors as sol_attn_fwd.
 */
int sol_attn_fwd_ws(const void* q, const void* k, const void* v, void* out, int B, int H, int N,
                    int D, int T, int Hl, int Wl, const float* rope_tab_dev, void* workspace,
                    size_t workspace_bytes, sol_stream_t stream);

/*
 * For callers that cannot allocate device memory -- code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc: the same
 * computation as sol_attn_fwd_ws (the same kernels, the same bits), on a
 * workspace the library holds itself instead of the caller's.  The workspace
 * is a static device array of SOL_NOALLOC_MAX_BYTES (256 MiB) on every GPU the
 * library runs on, held until the process ends; a call whose
 * sol_attn_workspace_bytes(B, H, N, D) exceeds it returns SOL_ERR_UNSUPPORTED
 * and launches nothing (e.g. B = 1, D = 128: H * ceil(N/32) * 32 <= 524,288,
 * such as 24 heads of 12,480 tokens).  The call allocates and frees nothing
 * (no hipMalloc, no allocating library routine).  Every call on one GPU uses
 * that GPU's one array: calls that overlap in time on one GPU (other streams,
 * other threads) race and must be serialised by the caller; calls in order on
 * one stream are safe.  Its contents between calls are unspecified (the
 * computation needs none cleared).  Other arguments, validation and errors as
 * sol_attn_fwd.
 */
#define SOL_NOALLOC_MAX_BYTES ((size_t)256 << 20)
int sol_attn_fwd_noalloc(const void* q, const void* k, const void* v, void* out, int B, int H,
                         int N, int D, int T, int Hl, int Wl, const float* rope_tab_dev,
                         sol_stream_t stream);

/*
 * Block-INT8 QKV records (Sec. 3.2, "Quantized communication"): the wire
 * format of the sequence-parallel QKV exchange.  One record per token and
 * head, 400 bytes (SOL_QKV_RECORD_BYTES):
 *   bytes   0..127  q codes, 128..255 k codes, 256..383 v codes: int8, two's
 *                   complement, dim d of a part at byte d of that part;
 *   bytes 384..395  scale codes, part p (0 q, 1 k, 2 v) dims [32g, 32g + 32)
 *                   at byte 384 + 4p + g: UE5M3 (unsigned, 5 exponent bits of
 *                   bias 15, 3 mantissa bits; exponent 0 subnormal, m 2^-17;
 *                   the encoder writes only the finite positive codes
 *                   0x01..0xF7 = 2^-17 .. 61440);
 *   bytes 396..399  zero.
 * Element value: bf16_RNE(code * scale).  Records are token-major: record
 * (b, n, h) at byte ((b N + n) H + h) * 400 -- the flat (tokens, heads,
 * record) layout the exchange delivers, heads being the receiver's head
 * share.  q and k in a record are as attention consumes them (normalised and
 * rotated): the records path applies no rotation of its own.
 *
 * sol_qkv_record_bytes: B * N * H * 400 (0 for invalid sizes).
 *
 * sol_qkv_encode: the sender's producer.  q, k, v: [B][H][N][D] bf16; q and k
 * are first RMS-normalised (q_gamma_dev, k_gamma_dev, eps as in
 * sol_qknorm_rope3d; NULL: not normalised) and rotated (rope_tab_dev, grid
 * T x Hl x Wl, as sol_qknorm_rope3d: the same bits), then each group of 32
 * values is quantised: scale s = the smallest finite positive UE5M3 value
 * with 127 s >= max |x| (0x01 for an all-zero group, 0xF7 when no code is
 * large enough), code = x / s rounded to nearest, ties to even, clamped to
 * [-127, 127].  Finite inputs.  rec must not overlap q, k or v.
 *
 * sol_qkv_encode_strided: the same, with q, k and v read where they lie
 * (Sec. 3.2: the stride-aware pack kernels read Q, K and V through their
 * existing strides, e.g. from packed QKV storage, and write the exchange
 * buffer in one pass): row (b, h, n) of each tensor starts at element
 * b stride_b + h stride_h + n stride_n of its pointer, its D values
 * contiguous.  Strides are non-negative multiples of 8 elements (rows stay
 * 16-byte aligned); a packed [B][N][3][H][D] buffer X is q = X, k = X + H D,
 * v = X + 2 H D with stride_b = 3 N H D, stride_h = D, stride_n = 3 H D.
 * sol_qkv_encode is this call with stride_b = H N D, stride_h = N D,
 * stride_n = D.  rec must not overlap the span of q, k or v.
 *
 * sol_qkv_decode: rec -> q, k, v ([B][H][N][D] bf16, element values as
 * above).  The outputs must not overlap rec or each other.
 *
 * sol_prepare_kv_records: sol_prepare_kv_ex with the keys and values taken
 * from the records (k and v parts) instead of bf16 tensors: keys key0 ..
 * key0 + N - 1 of a prepared sequence of n_kv keys, the same tile layout and
 * buffer sizes (sol_prepared_kv_bytes(B, H, n_kv, D)), no rotation.
 *
 * sol_attn_fwd_records: sol_attn_fwd_prepared_ex with the queries decoded
 * from the records (q parts) in the kernel's tile load: N query rows per
 * (b, h) against the n_kv prepared keys, no rotation or normalisation,
 * out [B][H][N][D] in out_format (SOL_OUT_BF16, SOL_OUT_FP8_E4M3 or
 * SOL_OUT_INT8_RECORDS).  Equal,
 * bit for bit, to sol_attn_fwd_prepared_ex on the decoded q (table NULL).
 *
 * All: D = 128; pointers 16-byte aligned device memory; 1 <= N <=
 * SOL_MAX_TOKENS; errors as the prepared path.
 */
#define SOL_QKV_RECORD_BYTES 400
#define SOL_OUT_RECORD_BYTES 144
size_t sol_qkv_record_bytes(int B, int H, int N);
int sol_qkv_encode(const void* q, const void* k, const void* v, void* rec, int B, int H, int N,
                   int D, int T, int Hl, int Wl, const float* rope_tab_dev,
                   const float* q_gamma_dev, const float* k_gamma_dev, float eps,
                   sol_stream_t stream);
int sol_qkv_encode_strided(const void* q, const void* k, const void* v, int64_t stride_b,
                           int64_t stride_h, int64_t stride_n, void* rec, int B, int H, int N, int D,
                           int T, int Hl, int Wl, const float* rope_tab_dev,
                           const float* q_gamma_dev, const float* k_gamma_dev, float eps,
                           sol_stream_t stream);
int sol_qkv_decode(const void* rec, void* q, void* k, void* v, int B, int H, int N, int D,
                   sol_stream_t stream);
int sol_prepare_kv_records(const void* rec, void* k_prep, void* v_prep, int B, int H, int N,
                           int key0, int n_kv, int D, sol_stream_t stream);
int sol_attn_fwd_records(const void* rec, const void* k_prep, const void* v_prep, void* out, int B,
                         int H, int N, int n_kv, int D, int out_format, sol_stream_t stream);

/*
 * Measurement aid: the dense matrix rate of this GPU at the attention
 * kernels' launch shape.  Launches `workgroups` workgroups of four waves (one
 * per SIMD, as the attention kernels run), each wave issuing iters * 16 fp16
 * MFMAs of 32 x 32 x 16 with fp32 accumulation on operands read once from
 * `operands` (8192 fp16 values, 16 KB, device memory): flops = workgroups *
 * 4 * iters * 16 * 32768.  `out` (workgroups * 256 floats, device) receives
 * per-thread sums so no product is skipped.  Time it with events on
 * `stream`: the datasheet peak assumes 2.4 GHz, while a long dense launch runs
 * at the clock the chip's power limit allows for such operands.
 * 1 <= workgroups <= 1 << 20, 1 <= iters <= 1 << 24; pointers 16-byte aligned.
 */
int sol_mfma_probe(const void* operands, float* out, int workgroups, int iters,
                   sol_stream_t stream);

/*
 * The current device's range status (SOL_RANGE_* bits raised since the last
 * clear) into *flags; clear != 0 resets it to 0.  The one call that
 * synchronises: it waits for all work on the current device first.  The
 * status is shared by every call on the device, whatever the stream or
 * thread.
 */
int sol_range_status(unsigned* flags, int clear);

/* Static description of a status code. */
const char* sol_status_string(int status);

/* Detail of the last failure on the calling thread ("" if none). */
const char* sol_last_error(void);

/* ABI version, major * 100 + minor. */
int sol_version(void);

#ifdef __cplusplus
}
#endif

#endif /* SOL_H */
