// C ABI front end of libsol.so: argument validation (before any HIP call),
// the host-side rotary table builder, launch and error mapping.
#include <stdarg.h>
#include <stdint.h>
#include <stdio.h>

#include <cmath>

#include "sol.h"
#include "sol_internal.h"

namespace {

thread_local char g_last_error[512] = "";

int fail(int status, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof g_last_error, fmt, ap);
  va_end(ap);
  return status;
}

int ok() {
  g_last_error[0] = '\0';
  return SOL_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

bool overlaps(const void* a, size_t na, const void* b, size_t nb) {
  const uintptr_t a0 = reinterpret_cast<uintptr_t>(a), b0 = reinterpret_cast<uintptr_t>(b);
  return a0 < b0 + nb && b0 < a0 + na;
}

// Common shape checks of the tensor entry points.
int check_shape(int B, int H, int N, int D, int T, int Hl, int Wl) {
  if (B < 1 || H < 1 || N < 1) return fail(SOL_ERR_INVALID_ARG, "B, H, N must be >= 1 (got %d, %d, %d)", B, H, N);
  if (T < 0 || Hl < 0 || Wl < 0) return fail(SOL_ERR_INVALID_ARG, "negative latent grid %dx%dx%d", T, Hl, Wl);
  if ((int64_t)T * Hl * Wl > N)
    return fail(SOL_ERR_INVALID_ARG, "latent grid %dx%dx%d holds more tokens than N=%d", T, Hl, Wl, N);
  if (D != sol::kHeadDim) return fail(SOL_ERR_UNSUPPORTED, "head dim %d not supported (only 128)", D);
  if (N > SOL_MAX_TOKENS) return fail(SOL_ERR_UNSUPPORTED, "N=%d exceeds %d", N, SOL_MAX_TOKENS);
  if ((int64_t)B * H > INT32_MAX) return fail(SOL_ERR_UNSUPPORTED, "B*H too large");
  return SOL_OK;
}

// The QK-normalisation arguments: no weights (eps ignored), or 16-byte
// aligned device weights with a finite eps >= 0.
int check_norm(const float* gamma, float eps) {
  if (!gamma) return SOL_OK;
  if (!aligned16(gamma)) return fail(SOL_ERR_INVALID_ARG, "gamma must be 16-byte aligned");
  if (!(eps >= 0.0f) || !std::isfinite(eps)) return fail(SOL_ERR_INVALID_ARG, "eps must be finite and >= 0");
  return SOL_OK;
}

// The rotary split: dt, dh, dw head dims turn with t, h, w; each a
// non-negative multiple of 8 (whole 16-byte chunks), together at most D; the
// remaining dims pass through.
int check_split(int D, int dt, int dh, int dw) {
  if (dt < 0 || dh < 0 || dw < 0 || dt % 8 || dh % 8 || dw % 8)
    return fail(SOL_ERR_INVALID_ARG, "rotary split %d/%d/%d: each must be a non-negative multiple of 8", dt, dh, dw);
  if ((int64_t)dt + dh + dw > D)
    return fail(SOL_ERR_INVALID_ARG, "rotary split %d/%d/%d exceeds the head dim %d", dt, dh, dw, D);
  return SOL_OK;
}

// The device table of a call: NULL when nothing rotates (an empty grid, or an
// empty split).
const float2* table_of(const float* rope_tab_dev, int T, int Hl, int Wl, int dt, int dh, int dw) {
  const bool rotates = (int64_t)T * Hl * Wl > 0 && dt + dh + dw > 0;
  return rotates ? reinterpret_cast<const float2*>(rope_tab_dev) : nullptr;
}

// Bytes of an attention output in out_format (0 for an unknown format).
size_t out_bytes(int B, int H, int N, int D, int out_format) {
  const size_t rows = (size_t)B * H * N;
  switch (out_format) {
    case SOL_OUT_BF16: return rows * D * 2;
    case SOL_OUT_FP8_E4M3: return rows * D;
    case SOL_OUT_INT8_RECORDS: return rows * SOL_OUT_RECORD_BYTES;
    default: return 0;
  }
}

// Common checks of the two block-sparse entry points.
int check_sparse(const void* q, const void* k_prep, int B, int H, int N, int D, int T, int Hl,
                 int Wl, int dt, int dh, int dw, const float* rope_tab_dev, const float* q_gamma_dev,
                 float eps, const void* workspace, size_t workspace_bytes) {
  if (!q || !k_prep) return fail(SOL_ERR_INVALID_ARG, "q and k_prep must not be NULL");
  int st = check_shape(B, H, N, D, T, Hl, Wl);
  if (st != SOL_OK) return st;
  if ((st = check_split(D, dt, dh, dw)) != SOL_OK) return st;
  if (N > sol::sparse_max_tokens())
    return fail(SOL_ERR_UNSUPPORTED, "block-sparse attention takes N <= %d (got %d)", sol::sparse_max_tokens(), N);
  if (!aligned16(q) || !aligned16(k_prep)) return fail(SOL_ERR_INVALID_ARG, "q and k_prep must be 16-byte aligned");
  if (rope_tab_dev && !aligned16(rope_tab_dev)) return fail(SOL_ERR_INVALID_ARG, "rope_tab_dev must be 16-byte aligned");
  st = check_norm(q_gamma_dev, eps);
  if (st != SOL_OK) return st;
  const size_t need = sol_sparse_workspace_bytes(B, H, N, D);
  if (!workspace) return fail(SOL_ERR_INVALID_ARG, "workspace is NULL");
  if (!aligned16(workspace)) return fail(SOL_ERR_INVALID_ARG, "workspace must be 16-byte aligned");
  if (workspace_bytes < need)
    return fail(SOL_ERR_INVALID_ARG, "workspace needs %zu bytes, got %zu", need, workspace_bytes);
  const size_t bytes = (size_t)B * H * N * D * 2;
  if (overlaps(workspace, need, q, bytes) || overlaps(workspace, need, k_prep, sol_prepared_kv_bytes(B, H, N, D)))
    return fail(SOL_ERR_INVALID_ARG, "workspace overlaps q or k_prep");
  return SOL_OK;
}

}  // namespace

int sol::set_error(int status, const char* msg) { return fail(status, "%s", msg); }

sol::SeqGrid sol::make_grid(int N, int T, int Hl, int Wl, int dt, int dh, int dw) {
  SeqGrid g;
  const int64_t nv = (int64_t)T * Hl * Wl;
  g.n = N;
  g.nt = (int)(N - nv);
  // An empty grid rotates nothing: every token is prefix; keep divisors valid.
  g.T = nv ? T : 1;
  g.Hl = nv ? Hl : 1;
  g.Wl = nv ? Wl : 1;
  g.hw = g.Hl * g.Wl;
  g.inv_hw = 1.0f / (float)g.hw;
  g.inv_wl = 1.0f / (float)g.Wl;
  g.c_t = dt / 8;
  g.c_h = g.c_t + dh / 8;
  g.c_w = g.c_h + dw / 8;
  g.s_t = dt / 2;
  g.s_h = dh / 2;
  g.s_w = dw / 2;
  g.tab_h = g.T * g.s_t;
  g.tab_w = g.tab_h + g.Hl * g.s_h;
  g.tab_pairs = g.tab_w + g.Wl * g.s_w;
  // row 0 of the first axis section that has one: angle 0 in every pair
  g.id_pair = dt ? 0 : dh ? g.tab_h : g.tab_w;
  return g;
}

extern "C" {

size_t sol_rope3d_table_floats_ex(int D, int T, int Hl, int Wl, int dt, int dh, int dw) {
  if (D <= 0 || D % 16 != 0 || T < 0 || Hl < 0 || Wl < 0) return 0;
  if (dt < 0 || dh < 0 || dw < 0 || dt % 8 || dh % 8 || dw % 8 || (int64_t)dt + dh + dw > D) return 0;
  // two planes (hi, then lo) of one (cos, sin) pair per rotary pair and position
  return 4 * ((size_t)T * (dt / 2) + (size_t)Hl * (dh / 2) + (size_t)Wl * (dw / 2));
}

size_t sol_rope3d_table_floats(int D, int T, int Hl, int Wl) {
  return sol_rope3d_table_floats_ex(D, T, Hl, Wl, D / 4, 3 * D / 8, 3 * D / 8);
}

int sol_rope3d_table_ex(float* host_tab, size_t n_floats, int D, int T, int Hl, int Wl, int dt,
                        int dh, int dw, double base) {
  if (D <= 0 || D % 16 != 0 || T < 0 || Hl < 0 || Wl < 0)
    return fail(SOL_ERR_INVALID_ARG, "bad table shape D=%d grid %dx%dx%d", D, T, Hl, Wl);
  int st = check_split(D, dt, dh, dw);
  if (st != SOL_OK) return st;
  const size_t need = sol_rope3d_table_floats_ex(D, T, Hl, Wl, dt, dh, dw);
  if (!host_tab && need) return fail(SOL_ERR_INVALID_ARG, "host_tab is NULL");
  if (n_floats < need) return fail(SOL_ERR_INVALID_ARG, "table needs %zu floats, got %zu", need, n_floats);
  if (!(base > 1.0) || !std::isfinite(base)) return fail(SOL_ERR_INVALID_ARG, "base must be finite and > 1");
  // Section for one axis of extent `len` whose chunk is `width` head dims wide:
  // row pos, pair i holds (cos, sin) of pos * base^(-2i/width), rounded to
  // fp32 in the hi plane; the lo plane, need / 2 floats on, holds what that
  // rounding lost, so that hi + lo carries the double to 48 bits.
  float* hi = host_tab;
  float* lo = host_tab + need / 2;
  auto put = [&](double x) {
    const float h = (float)x;
    *hi++ = h;
    *lo++ = (float)(x - (double)h);  // exact difference, rounded once
  };
  auto section = [&](int len, int width) {
    for (int pos = 0; pos < len; ++pos)
      for (int i = 0; i < width / 2; ++i) {
        const double phi = (double)pos * std::pow(base, -2.0 * i / (double)width);
        put(std::cos(phi));
        put(std::sin(phi));
      }
  };
  section(T, dt);
  section(Hl, dh);
  section(Wl, dw);
  return ok();
}

int sol_rope3d_table(float* host_tab, size_t n_floats, int D, int T, int Hl, int Wl, double base) {
  return sol_rope3d_table_ex(host_tab, n_floats, D, T, Hl, Wl, D / 4, 3 * D / 8, 3 * D / 8, base);
}

int sol_qknorm_rope3d(const void* x, void* y, int B, int H, int N, int D, int T, int Hl, int Wl,
                      int dt, int dh, int dw, const float* rope_tab_dev, const float* gamma_dev,
                      float eps, sol_stream_t stream) {
  if (!x || !y) return fail(SOL_ERR_INVALID_ARG, "x and y must not be NULL");
  int st = check_shape(B, H, N, D, T, Hl, Wl);
  if (st != SOL_OK) return st;
  if ((st = check_split(D, dt, dh, dw)) != SOL_OK) return st;
  if (!aligned16(x) || !aligned16(y)) return fail(SOL_ERR_INVALID_ARG, "x and y must be 16-byte aligned");
  const int64_t nv = (int64_t)T * Hl * Wl;
  if (nv > 0 && dt + dh + dw > 0 && !rope_tab_dev)
    return fail(SOL_ERR_INVALID_ARG, "rope_tab_dev is NULL for a non-empty grid and split");
  if (rope_tab_dev && !aligned16(rope_tab_dev)) return fail(SOL_ERR_INVALID_ARG, "rope_tab_dev must be 16-byte aligned");
  st = check_norm(gamma_dev, eps);
  if (st != SOL_OK) return st;
  const size_t bytes = (size_t)B * H * N * D * 2;
  if (x != y && overlaps(x, bytes, y, bytes)) return fail(SOL_ERR_INVALID_ARG, "x and y partially overlap");
  const sol::SeqGrid g = sol::make_grid(N, T, Hl, Wl, dt, dh, dw);
  hipError_t e = sol::launch_rope3d(static_cast<const uint16_t*>(x), static_cast<uint16_t*>(y),
                                    (int64_t)B * H * N, g, table_of(rope_tab_dev, T, Hl, Wl, dt, dh, dw),
                                    gamma_dev, eps, reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(SOL_ERR_HIP, "rope3d launch: %s", hipGetErrorString(e));
  return ok();
}

int sol_rope3d(const void* x, void* y, int B, int H, int N, int D, int T, int Hl, int Wl,
               const float* rope_tab_dev, sol_stream_t stream) {
  return sol_qknorm_rope3d(x, y, B, H, N, D, T, Hl, Wl, D / 4, 3 * D / 8, 3 * D / 8, rope_tab_dev,
                           nullptr, 0.0f, stream);
}

// sol_attn_fwd's schedule: chunks of whole (b, h) slabs, front to back, each
// through the prepared path with its prepared K and V held in the slabs of
// `out` after the chunk (not yet written); a chunk takes as many slabs as
// leave room for that, up to kMaxChunks chunks.  Of those chunks it keeps the
// leading ones that make the call fastest by a simple model: a launch over x
// workgroups takes ceil(x / 256) rounds on the 256 compute units, a round
// costs 1 on the prepared path and kFusedCost on the fused kernel (measured:
// 1.4 at 720p and at the low resolution), each chunk adds kChunkCost for its
// prepare pass and launches, and the slabs after the kept chunks run the
// fused kernel in one launch.  Returns the number of
// slabs the kept chunks cover and their sizes in chunk[].
constexpr int kMaxChunks = 64;
constexpr double kFusedCost = 1.4;
constexpr double kChunkCost = 0.1;
constexpr int kComputeUnits = 256;
static int attn_fwd_schedule(int B, int H, int N, int D, int (&chunk)[kMaxChunks]) {
  const int64_t S = (int64_t)B * H;
  const int64_t region = (int64_t)N * D * 2;                        // one slab of out
  const int64_t kv = 2 * sol::prepared_tile_elems(N) * 2;           // one slab of K and V tiles
  const int64_t nq = (N + sol::kFusedRows - 1) / sol::kFusedRows;   // workgroups per slab (both paths)
  auto rounds = [&](int64_t slabs) { return (double)((slabs * nq + kComputeUnits - 1) / kComputeUnits); };
  int64_t s = 0;
  int n = 0;
  for (; n < kMaxChunks && s < S; ++n) {
    // the largest c with c * kv <= (S - s - c) * region
    int64_t c = (S - s) * region / (kv + region);
    while (c > 0 && c * kv > (S - s - c) * region) --c;
    if (c == 0) break;
    chunk[n] = (int)c;
    s += c;
  }
  // keep the prefix of chunks with the lowest modelled time
  double best = kFusedCost * rounds(S), prefix = 0.0;
  int64_t covered = 0, best_covered = 0;
  for (int i = 0; i < n; ++i) {
    prefix += rounds(chunk[i]) + kChunkCost;
    covered += chunk[i];
    const double t = prefix + (covered < S ? kFusedCost * rounds(S - covered) : 0.0);
    if (t < best) {
      best = t;
      best_covered = covered;
    }
  }
  return (int)best_covered;
}

int sol_attn_fwd_plan(int B, int H, int N, int D) {
  int st = check_shape(B, H, N, D, 0, 0, 0);
  if (st != SOL_OK) return st;
  int chunk[kMaxChunks];
  return attn_fwd_schedule(B, H, N, D, chunk);
}

int sol_attn_fwd(const void* q, const void* k, const void* v, void* out, int B, int H, int N, int D,
                 int T, int Hl, int Wl, const float* rope_tab_dev, sol_stream_t stream) {
  if (!q || !k || !v || !out) return fail(SOL_ERR_INVALID_ARG, "q, k, v, out must not be NULL");
  int st = check_shape(B, H, N, D, T, Hl, Wl);
  if (st != SOL_OK) return st;
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(out))
    return fail(SOL_ERR_INVALID_ARG, "q, k, v, out must be 16-byte aligned");
  if (rope_tab_dev && !aligned16(rope_tab_dev)) return fail(SOL_ERR_INVALID_ARG, "rope_tab_dev must be 16-byte aligned");
  const size_t bytes = (size_t)B * H * N * D * 2;
  if (overlaps(out, bytes, q, bytes) || overlaps(out, bytes, k, bytes) || overlaps(out, bytes, v, bytes))
    return fail(SOL_ERR_INVALID_ARG, "out overlaps q, k or v");
  if (sol::attn_max_workgroups(N, B * H) > INT32_MAX) return fail(SOL_ERR_UNSUPPORTED, "grid too large");
  const int64_t nv = (int64_t)T * Hl * Wl;
  const float2* tab = nv > 0 ? reinterpret_cast<const float2*>(rope_tab_dev) : nullptr;
  const sol::SeqGrid g = sol::make_grid(N, T, Hl, Wl);
  const hipStream_t hs = reinterpret_cast<hipStream_t>(stream);
  const size_t slab = (size_t)N * D;  // elements of one (b, h) slab
  const uint16_t* qs = static_cast<const uint16_t*>(q);
  const uint16_t* ks = static_cast<const uint16_t*>(k);
  const uint16_t* vs = static_cast<const uint16_t*>(v);
  uint16_t* os = static_cast<uint16_t*>(out);
  const size_t kv_elems = (size_t)sol::prepared_tile_elems(N);  // per slab, K or V
  int chunk[kMaxChunks];
  const int covered = attn_fwd_schedule(B, H, N, D, chunk);
  int s = 0;
  for (int i = 0; s < covered; ++i) {
    const int c = chunk[i];
    // prepared K and V of slabs [s, s + c) in the out slabs from s + c on
    uint16_t* kp = os + (size_t)(s + c) * slab;
    uint16_t* vp = kp + (size_t)c * kv_elems;
    hipError_t e = sol::launch_prepare_kv(ks + s * slab, vs + s * slab, kp, vp, c, g, tab, 0, N, nullptr,
                                          0.0f, hs);
    if (e != hipSuccess) return fail(SOL_ERR_HIP, "attn_fwd (prepare) launch: %s", hipGetErrorString(e));
    e = sol::launch_attn_fwd_prepared(qs + s * slab, kp, vp, os + s * slab, c, g, N, tab, nullptr, 0.0f,
                                      SOL_OUT_BF16, nullptr, nullptr, 0, hs, nullptr, c);
    if (e != hipSuccess) return fail(SOL_ERR_HIP, "attn_fwd (attention) launch: %s", hipGetErrorString(e));
    s += c;
  }
  if (s < B * H) {
    hipError_t e = sol::launch_attn_fwd(qs + s * slab, ks + s * slab, vs + s * slab, os + s * slab,
                                        B * H - s, g, tab, hs);
    if (e != hipSuccess) return fail(SOL_ERR_HIP, "attn_fwd launch: %s", hipGetErrorString(e));
  }
  return ok();
}

size_t sol_prepared_kv_bytes(int B, int H, int N, int D) {
  if (B < 1 || H < 1 || N < 1 || D != 128 || N > SOL_MAX_TOKENS) return 0;
  return (size_t)B * H * (size_t)sol::prepared_tile_elems(N) * 2;
}

size_t sol_attn_workspace_bytes(int B, int H, int N, int D) {
  return 2 * sol_prepared_kv_bytes(B, H, N, D);
}

int sol_prepare_kv_ex(const void* k, const void* v, void* k_prep, void* v_prep, int B, int H,
                      int N, int key0, int n_kv, int D, int T, int Hl, int Wl, int dt, int dh,
                      int dw, const float* rope_tab_dev, const float* k_gamma_dev, float eps,
                      sol_stream_t stream) {
  if (!k || !v || !k_prep || !v_prep) return fail(SOL_ERR_INVALID_ARG, "k, v, k_prep, v_prep must not be NULL");
  int st = check_shape(B, H, N, D, T, Hl, Wl);
  if (st != SOL_OK) return st;
  if ((st = check_split(D, dt, dh, dw)) != SOL_OK) return st;
  if (n_kv < 1 || n_kv > SOL_MAX_TOKENS)
    return fail(n_kv < 1 ? SOL_ERR_INVALID_ARG : SOL_ERR_UNSUPPORTED, "n_kv=%d out of range", n_kv);
  if (key0 < 0 || (int64_t)key0 + N > n_kv)
    return fail(SOL_ERR_INVALID_ARG, "keys [%d, %lld) do not fit a sequence of n_kv=%d", key0,
                (long long)key0 + N, n_kv);
  if (!aligned16(k) || !aligned16(v) || !aligned16(k_prep) || !aligned16(v_prep))
    return fail(SOL_ERR_INVALID_ARG, "k, v, k_prep, v_prep must be 16-byte aligned");
  if (rope_tab_dev && !aligned16(rope_tab_dev)) return fail(SOL_ERR_INVALID_ARG, "rope_tab_dev must be 16-byte aligned");
  st = check_norm(k_gamma_dev, eps);
  if (st != SOL_OK) return st;
  const size_t bytes = (size_t)B * H * N * D * 2;
  const size_t pbytes = sol_prepared_kv_bytes(B, H, n_kv, D);
  if (overlaps(k_prep, pbytes, k, bytes) || overlaps(k_prep, pbytes, v, bytes) ||
      overlaps(v_prep, pbytes, k, bytes) || overlaps(v_prep, pbytes, v, bytes) ||
      overlaps(k_prep, pbytes, v_prep, pbytes))
    return fail(SOL_ERR_INVALID_ARG, "k_prep / v_prep overlap each other or k, v");
  const float2* tab = table_of(rope_tab_dev, T, Hl, Wl, dt, dh, dw);
  const sol::SeqGrid g = sol::make_grid(N, T, Hl, Wl, dt, dh, dw);
  hipError_t e = sol::launch_prepare_kv(static_cast<const uint16_t*>(k), static_cast<const uint16_t*>(v),
                                        static_cast<uint16_t*>(k_prep), static_cast<uint16_t*>(v_prep), B * H,
                                        g, tab, key0, n_kv, k_gamma_dev, eps,
                                        reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(SOL_ERR_HIP, "prepare_kv launch: %s", hipGetErrorString(e));
  return ok();
}

int sol_prepare_kv(const void* k, const void* v, void* k_prep, void* v_prep, int B, int H, int N,
                   int D, int T, int Hl, int Wl, const float* rope_tab_dev, sol_stream_t stream) {
  return sol_prepare_kv_ex(k, v, k_prep, v_prep, B, H, N, 0, N, D, T, Hl, Wl, D / 4, 3 * D / 8,
                           3 * D / 8, rope_tab_dev, nullptr, 0.0f, stream);
}

int sol_attn_fwd_prepared_ex(const void* q, const void* k_prep, const void* v_prep, void* out,
                             int B, int H, int N, int n_kv, int D, int T, int Hl, int Wl, int dt,
                             int dh, int dw, const float* rope_tab_dev, const float* q_gamma_dev,
                             float eps, int out_format, sol_stream_t stream) {
  if (!q || !k_prep || !v_prep || !out) return fail(SOL_ERR_INVALID_ARG, "q, k_prep, v_prep, out must not be NULL");
  int st = check_shape(B, H, N, D, T, Hl, Wl);
  if (st != SOL_OK) return st;
  if ((st = check_split(D, dt, dh, dw)) != SOL_OK) return st;
  if (n_kv < 1 || n_kv > SOL_MAX_TOKENS)
    return fail(n_kv < 1 ? SOL_ERR_INVALID_ARG : SOL_ERR_UNSUPPORTED, "n_kv=%d out of range", n_kv);
  if (!aligned16(q) || !aligned16(k_prep) || !aligned16(v_prep) || !aligned16(out))
    return fail(SOL_ERR_INVALID_ARG, "q, k_prep, v_prep, out must be 16-byte aligned");
  if (rope_tab_dev && !aligned16(rope_tab_dev)) return fail(SOL_ERR_INVALID_ARG, "rope_tab_dev must be 16-byte aligned");
  st = check_norm(q_gamma_dev, eps);
  if (st != SOL_OK) return st;
  const size_t obytes = out_bytes(B, H, N, D, out_format);
  if (obytes == 0) return fail(SOL_ERR_INVALID_ARG, "unknown out_format %d", out_format);
  const size_t bytes = (size_t)B * H * N * D * 2;
  const size_t pbytes = sol_prepared_kv_bytes(B, H, n_kv, D);
  if (overlaps(out, obytes, q, bytes) || overlaps(out, obytes, k_prep, pbytes) || overlaps(out, obytes, v_prep, pbytes))
    return fail(SOL_ERR_INVALID_ARG, "out overlaps q, k_prep or v_prep");
  if (sol::attn_max_workgroups(N, B * H) > INT32_MAX) return fail(SOL_ERR_UNSUPPORTED, "grid too large");
  const float2* tab = table_of(rope_tab_dev, T, Hl, Wl, dt, dh, dw);
  const sol::SeqGrid g = sol::make_grid(N, T, Hl, Wl, dt, dh, dw);
  hipError_t e = sol::launch_attn_fwd_prepared(static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k_prep),
                                               static_cast<const uint16_t*>(v_prep), out, B * H, g, n_kv, tab,
                                               q_gamma_dev, eps, out_format, nullptr, nullptr, 0,
                                               reinterpret_cast<hipStream_t>(stream), nullptr, H);
  if (e != hipSuccess) return fail(SOL_ERR_HIP, "attn_fwd_prepared launch: %s", hipGetErrorString(e));
  return ok();
}

int sol_attn_fwd_prepared(const void* q, const void* k_prep, const void* v_prep, void* out, int B,
                          int H, int N, int D, int T, int Hl, int Wl, const float* rope_tab_dev,
                          sol_stream_t stream) {
  return sol_attn_fwd_prepared_ex(q, k_prep, v_prep, out, B, H, N, N, D, T, Hl, Wl, D / 4, 3 * D / 8,
                                  3 * D / 8, rope_tab_dev, nullptr, 0.0f, SOL_OUT_BF16, stream);
}

size_t sol_sparse_workspace_bytes(int B, int H, int N, int D) {
  if (B < 1 || H < 1 || N < 1 || D != sol::kHeadDim || N > sol::sparse_max_tokens()) return 0;
  if ((int64_t)B * H > INT32_MAX) return 0;
  size_t off[4];
  return sol::sparse_workspace_offsets(B * H, N, off);
}

int sol_sparse_route(const void* q, const void* k_prep, int B, int H, int N, int D, int T, int Hl,
                     int Wl, int dt, int dh, int dw, const float* rope_tab_dev,
                     const float* q_gamma_dev, float eps, float tau, void* workspace,
                     size_t workspace_bytes, sol_stream_t stream) {
  int st = check_sparse(q, k_prep, B, H, N, D, T, Hl, Wl, dt, dh, dw, rope_tab_dev, q_gamma_dev, eps,
                        workspace, workspace_bytes);
  if (st != SOL_OK) return st;
  if (!std::isfinite(tau)) return fail(SOL_ERR_INVALID_ARG, "tau must be finite");
  const float2* tab = table_of(rope_tab_dev, T, Hl, Wl, dt, dh, dw);
  const sol::SeqGrid g = sol::make_grid(N, T, Hl, Wl, dt, dh, dw);
  hipError_t e = sol::launch_sparse_route(static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k_prep),
                                          B * H, g, tab, q_gamma_dev, eps, tau, workspace,
                                          reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(SOL_ERR_HIP, "sparse_route launch: %s", hipGetErrorString(e));
  return ok();
}

int sol_attn_fwd_sparse(const void* q, const void* k_prep, const void* v_prep, void* out, int B,
                        int H, int N, int D, int T, int Hl, int Wl, int dt, int dh, int dw,
                        const float* rope_tab_dev, const float* q_gamma_dev, float eps,
                        const void* workspace, size_t workspace_bytes, int out_format,
                        sol_stream_t stream) {
  int st = check_sparse(q, k_prep, B, H, N, D, T, Hl, Wl, dt, dh, dw, rope_tab_dev, q_gamma_dev, eps,
                        workspace, workspace_bytes);
  if (st != SOL_OK) return st;
  if (!v_prep || !out) return fail(SOL_ERR_INVALID_ARG, "v_prep and out must not be NULL");
  if (!aligned16(v_prep) || !aligned16(out)) return fail(SOL_ERR_INVALID_ARG, "v_prep and out must be 16-byte aligned");
  const size_t obytes = out_bytes(B, H, N, D, out_format);
  if (obytes == 0) return fail(SOL_ERR_INVALID_ARG, "unknown out_format %d", out_format);
  const size_t bytes = (size_t)B * H * N * D * 2;
  const size_t pbytes = sol_prepared_kv_bytes(B, H, N, D);
  const size_t need = sol_sparse_workspace_bytes(B, H, N, D);
  if (overlaps(out, obytes, q, bytes) || overlaps(out, obytes, k_prep, pbytes) ||
      overlaps(out, obytes, v_prep, pbytes) || overlaps(out, obytes, workspace, need))
    return fail(SOL_ERR_INVALID_ARG, "out overlaps q, k_prep, v_prep or the workspace");
  if (sol::attn_max_workgroups(N, B * H) > INT32_MAX) return fail(SOL_ERR_UNSUPPORTED, "grid too large");
  const float2* tab = table_of(rope_tab_dev, T, Hl, Wl, dt, dh, dw);
  const sol::SeqGrid g = sol::make_grid(N, T, Hl, Wl, dt, dh, dw);
  size_t off[4];
  sol::sparse_workspace_offsets(B * H, N, off);
  const char* ws = static_cast<const char*>(workspace);
  hipError_t e = sol::launch_attn_fwd_prepared(
      static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k_prep), static_cast<const uint16_t*>(v_prep),
      out, B * H, g, N, tab, q_gamma_dev, eps, out_format,
      reinterpret_cast<const uint16_t*>(ws + off[1]), reinterpret_cast<const int*>(ws + off[0]),
      (N + 127) / 128, reinterpret_cast<hipStream_t>(stream), nullptr, H);
  if (e != hipSuccess) return fail(SOL_ERR_HIP, "attn_fwd_sparse launch: %s", hipGetErrorString(e));
  return ok();
}

int sol_attn_fwd_ws(const void* q, const void* k, const void* v, void* out, int B, int H, int N,
                    int D, int T, int Hl, int Wl, const float* rope_tab_dev, void* workspace,
                    size_t workspace_bytes, sol_stream_t stream) {
  if (!q || !k || !v || !out) return fail(SOL_ERR_INVALID_ARG, "q, k, v, out must not be NULL");
  int st = check_shape(B, H, N, D, T, Hl, Wl);
  if (st != SOL_OK) return st;
  const size_t bytes = (size_t)B * H * N * D * 2;
  const size_t need = sol_attn_workspace_bytes(B, H, N, D);
  if (!workspace) return fail(SOL_ERR_INVALID_ARG, "workspace is NULL");
  if (!aligned16(workspace)) return fail(SOL_ERR_INVALID_ARG, "workspace must be 16-byte aligned");
  if (workspace_bytes < need)
    return fail(SOL_ERR_INVALID_ARG, "workspace needs %zu bytes, got %zu", need, workspace_bytes);
  if (overlaps(workspace, need, q, bytes) || overlaps(workspace, need, k, bytes) ||
      overlaps(workspace, need, v, bytes) || overlaps(workspace, need, out, bytes))
    return fail(SOL_ERR_INVALID_ARG, "workspace overlaps q, k, v or out");
  if (overlaps(out, bytes, q, bytes) || overlaps(out, bytes, k, bytes) || overlaps(out, bytes, v, bytes))
    return fail(SOL_ERR_INVALID_ARG, "out overlaps q, k or v");
  uint16_t* k_prep = static_cast<uint16_t*>(workspace);
  uint16_t* v_prep = k_prep + sol_prepared_kv_bytes(B, H, N, D) / 2;
  st = sol_prepare_kv(k, v, k_prep, v_prep, B, H, N, D, T, Hl, Wl, rope_tab_dev, stream);
  if (st != SOL_OK) return st;
  return sol_attn_fwd_prepared(q, k_prep, v_prep, out, B, H, N, D, T, Hl, Wl, rope_tab_dev, stream);
}

size_t sol_qkv_record_bytes(int B, int H, int N) {
  if (B < 1 || H < 1 || N < 1 || N > SOL_MAX_TOKENS) return 0;
  const int64_t n_rec = (int64_t)B * N * H;
  if ((n_rec + 3) / 4 > INT32_MAX) return 0;
  return (size_t)n_rec * SOL_QKV_RECORD_BYTES;
}

int sol_qkv_encode(const void* q, const void* k, const void* v, void* rec, int B, int H, int N,
                   int D, int T, int Hl, int Wl, const float* rope_tab_dev,
                   const float* q_gamma_dev, const float* k_gamma_dev, float eps,
                   sol_stream_t stream) {
  return sol_qkv_encode_strided(q, k, v, (int64_t)H * N * D, (int64_t)N * D, D, rec, B, H, N, D, T, Hl,
                                Wl, rope_tab_dev, q_gamma_dev, k_gamma_dev, eps, stream);
}

int sol_qkv_encode_strided(const void* q, const void* k, const void* v, int64_t stride_b,
                           int64_t stride_h, int64_t stride_n, void* rec, int B, int H, int N, int D,
                           int T, int Hl, int Wl, const float* rope_tab_dev,
                           const float* q_gamma_dev, const float* k_gamma_dev, float eps,
                           sol_stream_t stream) {
  if (!q || !k || !v || !rec) return fail(SOL_ERR_INVALID_ARG, "q, k, v, rec must not be NULL");
  int st = check_shape(B, H, N, D, T, Hl, Wl);
  if (st != SOL_OK) return st;
  if (stride_b < 0 || stride_h < 0 || stride_n < 0 || stride_b % 8 || stride_h % 8 || stride_n % 8)
    return fail(SOL_ERR_INVALID_ARG, "strides must be non-negative multiples of 8 elements");
  // the extent each tensor spans: its last row's offset plus one row
  const int64_t span = ((int64_t)(B - 1) * stride_b + (int64_t)(H - 1) * stride_h +
                        (int64_t)(N - 1) * stride_n + D) * 2;
  const size_t rbytes = sol_qkv_record_bytes(B, H, N);
  if (rbytes == 0) return fail(SOL_ERR_UNSUPPORTED, "too many records");
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(rec))
    return fail(SOL_ERR_INVALID_ARG, "q, k, v, rec must be 16-byte aligned");
  if (rope_tab_dev && !aligned16(rope_tab_dev)) return fail(SOL_ERR_INVALID_ARG, "rope_tab_dev must be 16-byte aligned");
  if ((st = check_norm(q_gamma_dev, eps)) != SOL_OK || (st = check_norm(k_gamma_dev, eps)) != SOL_OK)
    return st;
  if (overlaps(rec, rbytes, q, span) || overlaps(rec, rbytes, k, span) || overlaps(rec, rbytes, v, span))
    return fail(SOL_ERR_INVALID_ARG, "rec overlaps q, k or v");
  const int64_t nv = (int64_t)T * Hl * Wl;
  const float2* tab = nv > 0 ? reinterpret_cast<const float2*>(rope_tab_dev) : nullptr;
  hipError_t e = sol::launch_qkv_encode(static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k),
                                        static_cast<const uint16_t*>(v), static_cast<uint8_t*>(rec), B, H,
                                        sol::make_grid(N, T, Hl, Wl), tab, q_gamma_dev, k_gamma_dev, eps,
                                        stride_b, stride_h, stride_n, reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(SOL_ERR_HIP, "qkv_encode launch: %s", hipGetErrorString(e));
  return ok();
}

int sol_qkv_decode(const void* rec, void* q, void* k, void* v, int B, int H, int N, int D,
                   sol_stream_t stream) {
  if (!q || !k || !v || !rec) return fail(SOL_ERR_INVALID_ARG, "rec, q, k, v must not be NULL");
  int st = check_shape(B, H, N, D, 0, 0, 0);
  if (st != SOL_OK) return st;
  const size_t rbytes = sol_qkv_record_bytes(B, H, N);
  if (rbytes == 0) return fail(SOL_ERR_UNSUPPORTED, "too many records");
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(rec))
    return fail(SOL_ERR_INVALID_ARG, "rec, q, k, v must be 16-byte aligned");
  const size_t bytes = (size_t)B * H * N * D * 2;
  if (overlaps(rec, rbytes, q, bytes) || overlaps(rec, rbytes, k, bytes) || overlaps(rec, rbytes, v, bytes) ||
      overlaps(q, bytes, k, bytes) || overlaps(q, bytes, v, bytes) || overlaps(k, bytes, v, bytes))
    return fail(SOL_ERR_INVALID_ARG, "q, k, v overlap rec or each other");
  hipError_t e = sol::launch_qkv_decode(static_cast<const uint8_t*>(rec), static_cast<uint16_t*>(q),
                                        static_cast<uint16_t*>(k), static_cast<uint16_t*>(v), B, H, N,
                                        reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(SOL_ERR_HIP, "qkv_decode launch: %s", hipGetErrorString(e));
  return ok();
}

int sol_prepare_kv_records(const void* rec, void* k_prep, void* v_prep, int B, int H, int N,
                           int key0, int n_kv, int D, sol_stream_t stream) {
  if (!rec || !k_prep || !v_prep) return fail(SOL_ERR_INVALID_ARG, "rec, k_prep, v_prep must not be NULL");
  int st = check_shape(B, H, N, D, 0, 0, 0);
  if (st != SOL_OK) return st;
  const size_t rbytes = sol_qkv_record_bytes(B, H, N);
  if (rbytes == 0) return fail(SOL_ERR_UNSUPPORTED, "too many records");
  if (n_kv < 1 || n_kv > SOL_MAX_TOKENS)
    return fail(n_kv < 1 ? SOL_ERR_INVALID_ARG : SOL_ERR_UNSUPPORTED, "n_kv=%d out of range", n_kv);
  if (key0 < 0 || (int64_t)key0 + N > n_kv)
    return fail(SOL_ERR_INVALID_ARG, "keys [%d, %lld) do not fit a sequence of n_kv=%d", key0,
                (long long)key0 + N, n_kv);
  if (!aligned16(rec) || !aligned16(k_prep) || !aligned16(v_prep))
    return fail(SOL_ERR_INVALID_ARG, "rec, k_prep, v_prep must be 16-byte aligned");
  const size_t pbytes = sol_prepared_kv_bytes(B, H, n_kv, D);
  if (overlaps(k_prep, pbytes, rec, rbytes) || overlaps(v_prep, pbytes, rec, rbytes) ||
      overlaps(k_prep, pbytes, v_prep, pbytes))
    return fail(SOL_ERR_INVALID_ARG, "k_prep / v_prep overlap each other or rec");
  hipError_t e = sol::launch_prepare_kv_records(static_cast<const uint8_t*>(rec), static_cast<uint16_t*>(k_prep),
                                                static_cast<uint16_t*>(v_prep), B, H, N, key0, n_kv,
                                                reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(SOL_ERR_HIP, "prepare_kv_records launch: %s", hipGetErrorString(e));
  return ok();
}

int sol_attn_fwd_records(const void* rec, const void* k_prep, const void* v_prep, void* out, int B,
                         int H, int N, int n_kv, int D, int out_format, sol_stream_t stream) {
  if (!rec || !k_prep || !v_prep || !out) return fail(SOL_ERR_INVALID_ARG, "rec, k_prep, v_prep, out must not be NULL");
  int st = check_shape(B, H, N, D, 0, 0, 0);
  if (st != SOL_OK) return st;
  const size_t rbytes = sol_qkv_record_bytes(B, H, N);
  if (rbytes == 0) return fail(SOL_ERR_UNSUPPORTED, "too many records");
  if (n_kv < 1 || n_kv > SOL_MAX_TOKENS)
    return fail(n_kv < 1 ? SOL_ERR_INVALID_ARG : SOL_ERR_UNSUPPORTED, "n_kv=%d out of range", n_kv);
  if (!aligned16(rec) || !aligned16(k_prep) || !aligned16(v_prep) || !aligned16(out))
    return fail(SOL_ERR_INVALID_ARG, "rec, k_prep, v_prep, out must be 16-byte aligned");
  const size_t obytes = out_bytes(B, H, N, D, out_format);
  if (obytes == 0) return fail(SOL_ERR_INVALID_ARG, "unknown out_format %d", out_format);
  const size_t pbytes = sol_prepared_kv_bytes(B, H, n_kv, D);
  if (overlaps(out, obytes, rec, rbytes) || overlaps(out, obytes, k_prep, pbytes) || overlaps(out, obytes, v_prep, pbytes))
    return fail(SOL_ERR_INVALID_ARG, "out overlaps rec, k_prep or v_prep");
  if (sol::attn_max_workgroups(N, B * H) > INT32_MAX) return fail(SOL_ERR_UNSUPPORTED, "grid too large");
  hipError_t e = sol::launch_attn_fwd_prepared(nullptr, static_cast<const uint16_t*>(k_prep),
                                               static_cast<const uint16_t*>(v_prep), out, B * H,
                                               sol::make_grid(N, 0, 0, 0), n_kv, nullptr, nullptr, 0.0f,
                                               out_format, nullptr, nullptr, 0,
                                               reinterpret_cast<hipStream_t>(stream),
                                               static_cast<const uint8_t*>(rec), H);
  if (e != hipSuccess) return fail(SOL_ERR_HIP, "attn_fwd_records launch: %s", hipGetErrorString(e));
  return ok();
}

int sol_mfma_probe(const void* operands, float* out, int workgroups, int iters, sol_stream_t stream) {
  if (!operands || !out) return fail(SOL_ERR_INVALID_ARG, "operands, out must not be NULL");
  if (workgroups < 1 || workgroups > (1 << 20) || iters < 1 || iters > (1 << 24))
    return fail(SOL_ERR_INVALID_ARG, "workgroups %d or iters %d out of range", workgroups, iters);
  if (!aligned16(operands) || !aligned16(out)) return fail(SOL_ERR_INVALID_ARG, "operands, out must be 16-byte aligned");
  if (overlaps(out, (size_t)workgroups * 256 * 4, operands, 16384))
    return fail(SOL_ERR_INVALID_ARG, "out overlaps operands");
  hipError_t e = sol::launch_mfma_probe(static_cast<const uint16_t*>(operands), out, workgroups, iters,
                                        reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(SOL_ERR_HIP, "mfma_probe launch: %s", hipGetErrorString(e));
  return ok();
}

int sol_range_status(unsigned* flags, int clear) {
  if (!flags) return fail(SOL_ERR_INVALID_ARG, "flags must not be NULL");
  hipError_t e = sol::range_status(flags, clear != 0);
  if (e != hipSuccess) return fail(SOL_ERR_HIP, "range status: %s", hipGetErrorString(e));
  return ok();
}

const char* sol_status_string(int status) {
  switch (status) {
    case SOL_OK: return "ok";
    case SOL_ERR_INVALID_ARG: return "invalid argument";
    case SOL_ERR_UNSUPPORTED: return "unsupported configuration";
    case SOL_ERR_HIP: return "HIP runtime error";
    default: return "unknown status";
  }
}

const char* sol_last_error(void) { return g_last_error; }

int sol_version(void) { return 200; }

}  // extern "C"
