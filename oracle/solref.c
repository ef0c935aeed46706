/*
 * solref.c -- CPU oracle for 3D-RoPE + full softmax attention.
 *
 * TEST INFRASTRUCTURE, NOT PRODUCT CODE.  Only the test suite, the smoke check
 * and the benchmark's CPU-baseline leg may load this library.  It shares no
 * code, header, table or constant generator with the HIP library: its own
 * trigonometry, its own token indexing, its own bf16 rounding.
 *
 * What it computes (all arithmetic in IEEE double):
 *
 *   The video DiT's spatio-temporal self-attention (Sec. 3.2 "Optimized
 *   attention collectives": the SDPA term that dominates the denoising step;
 *   Sec. 3.4: its cost grows with the square of the token count) applied to
 *   queries and keys that first pass through the partial/3D rotary embedding
 *   of Sec. 3.5 (fusion group 2, "QK normalization with partial RoPE").  The
 *   normalization half is optional: when a weight vector gamma is given, each
 *   head's D-vector is first RMS-normalised,
 *     x <- gamma * x / sqrt(mean_d(x_d^2) + eps),
 *   over every token (prefix included), then rotated; the bf16 input is the
 *   rounding point the paper keeps ahead of QK normalization (Sec. 3.5,
 *   "LoRA fusion"), and nothing is rounded between normalization and rotation.
 *
 *   Sequence packing (Sec. 3.4 "Safety rails"): the Nt = N - T*Hl*Wl leading
 *   tokens are a prefix (text) that is not rotated; token n >= Nt is the
 *   video latent at r = n - Nt, raster order t-major: t = r / (Hl*Wl),
 *   h = (r / Wl) mod Hl, w = r mod Wl.
 *
 *   Rotary embedding: head dims [0,dt) carry t, [dt,dt+dh) carry h,
 *   [dt+dh,dt+dh+dw) carry w, the rest pass through.  Inside an axis chunk of
 *   width d, the pair (2i, 2i+1) is the complex number x_{2i} + j x_{2i+1},
 *   multiplied by exp(j * pos * base^(-2i/d)).
 *
 *   Rounding point ("contract" mode, the default): the rotated (and, with
 *   gamma, normalised) q and k are rounded to bf16 (round to nearest, ties to
 *   even) once, as any bf16 matrix unit must consume them.  contract = 0 keeps
 *   them in double (diagnostic).
 *
 *   Attention per (b, h, query i), the plain two-pass definition:
 *     s_j = <q_i, k_j> / sqrt(D)               for every key j < N
 *     m   = max_j s_j
 *     p_j = exp(s_j - m),  l = sum_j p_j
 *     o_i = (sum_j p_j v_j) / l
 *
 * Tensors: bf16 bit patterns (uint16), contiguous [B][H][N][D].
 */
#define _GNU_SOURCE
#include <math.h>
#include <pthread.h>
#include <sched.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* bf16 bit pattern -> double (exact). */
static double bf16_to_double(uint16_t b) {
  uint32_t u = (uint32_t)b << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return (double)f;
}

/* double -> bf16 bit pattern, round to nearest, ties to even, computed from
 * the double directly (no intermediate float rounding).  NaN -> quiet NaN. */
static uint16_t double_to_bf16(double x) {
  if (isnan(x)) return 0x7fc0;
  uint16_t sign = signbit(x) ? 0x8000 : 0;
  double a = fabs(x);
  if (a == 0.0) return sign;
  if (isinf(a)) return sign | 0x7f80;
  /* bf16: 8 significant bits.  Find e with 2^e <= a < 2^(e+1). */
  int e;
  (void)frexp(a, &e); /* a = f * 2^e with f in [0.5, 1) */
  e -= 1;             /* now 2^e <= a < 2^(e+1) */
  if (e < -126) e = -126;   /* subnormal range: fixed quantum 2^-133 */
  double quantum = ldexp(1.0, e - 7);
  double n = a / quantum;   /* exact: power-of-two division */
  double fl = floor(n);
  double rem = n - fl;
  if (rem > 0.5 || (rem == 0.5 && fmod(fl, 2.0) != 0.0)) fl += 1.0;
  double r = fl * quantum;
  if (r >= ldexp(1.0, 128)) return sign | 0x7f80; /* overflow to inf */
  float rf = (float)r; /* exact: r has at most 8 significant bits */
  uint32_t u;
  memcpy(&u, &rf, sizeof u);
  return sign | (uint16_t)(u >> 16);
}

void solref_round_bf16(const double* x, uint16_t* y, int64_t n) {
  for (int64_t i = 0; i < n; ++i) y[i] = double_to_bf16(x[i]);
}

/* double -> FP8 E4M3 code (the OCP "E4M3FN" format: sign, 4 exponent bits of
 * bias 7, 3 mantissa bits; no infinities; codes 0x7F/0xFF are NaN; largest
 * finite value 448, smallest subnormal 2^-9), round to nearest, ties to even,
 * saturating: every |x| >= 448 (infinities included) gives +-448.  This is the
 * raw E4M3 output the paper's attention hands to the next GEMM with unit
 * scales (Sec. 3.3, "Joint optimization with quantized communication"). */
static uint8_t double_to_e4m3(double x) {
  if (isnan(x)) return 0x7f;
  uint8_t sign = signbit(x) ? 0x80 : 0;
  double a = fabs(x);
  if (a >= 448.0) return sign | 0x7e;
  if (a == 0.0) return sign;
  int e;
  (void)frexp(a, &e);
  e -= 1;                  /* 2^e <= a < 2^(e+1) */
  if (e < -6) e = -6;      /* subnormal range: fixed quantum 2^-9 */
  double quantum = ldexp(1.0, e - 3);
  double n = a / quantum;  /* exact: power-of-two division */
  double fl = floor(n);
  double rem = n - fl;
  if (rem > 0.5 || (rem == 0.5 && ((int64_t)fl & 1))) fl += 1.0;
  int m = (int)fl;         /* significand in units of the quantum: 0..16 */
  if (m == 16) {           /* rounded up into the next binade */
    m = 8;
    e += 1;
  }
  if (m < 8) return sign | (uint8_t)m;  /* subnormal (e == -6) */
  return sign | (uint8_t)(((e + 7) << 3) | (m - 8));
}

void solref_round_e4m3(const double* x, uint8_t* y, int64_t n) {
  for (int64_t i = 0; i < n; ++i) y[i] = double_to_e4m3(x[i]);
}

/* Position of token n on each axis; returns 0 for a prefix (unrotated) token. */
static int token_position(int64_t n, int N, int T, int Hl, int Wl, int* pt, int* ph, int* pw) {
  int64_t nv = (int64_t)T * Hl * Wl;
  int64_t nt = (int64_t)N - nv;
  if (nv == 0) return 0; /* empty grid: every token is prefix */
  if (n < nt) return 0;
  int64_t r = n - nt;
  *pt = (int)(r / ((int64_t)Hl * Wl));
  *ph = (int)((r / Wl) % Hl);
  *pw = (int)(r % Wl);
  (void)T;
  return 1;
}

/* Rotate one D-vector (in place, double) by the 3D rotary embedding at
 * (pt, ph, pw).  Axis chunks are [0,dt), [dt,dt+dh), [dt+dh,dt+dh+dw). */
static void rotate_vector(double* x, int D, int dt, int dh, int dw, double base,
                          int pt, int ph, int pw) {
  const int widths[3] = {dt, dh, dw};
  const int pos[3] = {pt, ph, pw};
  int off = 0;
  for (int a = 0; a < 3; ++a) {
    int d = widths[a];
    for (int i = 0; i < d / 2; ++i) {
      double theta = pow(base, -2.0 * i / (double)d);
      double phi = (double)pos[a] * theta;
      double c = cos(phi), s = sin(phi);
      double re = x[off + 2 * i], im = x[off + 2 * i + 1];
      x[off + 2 * i] = re * c - im * s;
      x[off + 2 * i + 1] = re * s + im * c;
    }
    off += d;
  }
  (void)D;
}

/* RMS normalisation of one D-vector (in place, double): the root mean square
 * over the head's D entries, eps added under the root, then the per-dimension
 * weight gamma[d]. */
static void rms_normalize(double* x, int D, const double* gamma, double eps) {
  double ss = 0.0;
  for (int d = 0; d < D; ++d) ss += x[d] * x[d];
  const double inv = 1.0 / sqrt(ss / (double)D + eps);
  for (int d = 0; d < D; ++d) x[d] = x[d] * inv * gamma[d];
}

/* One row of a bf16 tensor [BH][N][D] -> doubles: normalised first when gamma
 * is given, then rotated.  If contract and either step changed the row, the
 * result is rounded to bf16 (then widened back, exactly). */
static void rotate_row(const uint16_t* src, double* dst, int64_t n, int N, int D,
                       int T, int Hl, int Wl, int dt, int dh, int dw, double base,
                       int use_rope, int contract, const double* gamma, double eps) {
  for (int d = 0; d < D; ++d) dst[d] = bf16_to_double(src[d]);
  int changed = 0;
  if (gamma) {
    rms_normalize(dst, D, gamma, eps);
    changed = 1;
  }
  int pt, ph, pw;
  if (use_rope && token_position(n, N, T, Hl, Wl, &pt, &ph, &pw)) {
    rotate_vector(dst, D, dt, dh, dw, base, pt, ph, pw);
    changed = 1;
  }
  if (contract && changed)
    for (int d = 0; d < D; ++d) dst[d] = bf16_to_double(double_to_bf16(dst[d]));
}

/* Rotation in double, no rounding: x, y are double [rows][D]; row r is token r mod N. */
void solref_rope3d_f64(const double* x, double* y, int64_t rows, int N, int D,
                       int T, int Hl, int Wl, int dt, int dh, int dw, double base) {
  for (int64_t r = 0; r < rows; ++r) {
    int64_t n = r % N;
    for (int d = 0; d < D; ++d) y[r * D + d] = x[r * D + d];
    int pt, ph, pw;
    if (token_position(n, N, T, Hl, Wl, &pt, &ph, &pw))
      rotate_vector(y + r * D, D, dt, dh, dw, base, pt, ph, pw);
  }
}

/* Contract-mode rotation of a bf16 tensor: rotate in double, round once to bf16. */
void solref_rope3d(const uint16_t* x, uint16_t* y, int64_t rows, int N, int D,
                   int T, int Hl, int Wl, int dt, int dh, int dw, double base) {
  double* buf = (double*)malloc(sizeof(double) * (size_t)D);
  for (int64_t r = 0; r < rows; ++r) {
    int64_t n = r % N;
    rotate_row(x + r * D, buf, n, N, D, T, Hl, Wl, dt, dh, dw, base, 1, 0, NULL, 0.0);
    for (int d = 0; d < D; ++d) y[r * D + d] = double_to_bf16(buf[d]);
  }
  free(buf);
}

/* Contract-mode QK normalisation + rotation of a bf16 tensor: normalise with
 * gamma[D] and eps, rotate, all in double, round once to bf16.  rope = 0
 * normalises only.  contract = 0 writes the doubles to yf (diagnostic) and
 * leaves y untouched; y or yf may be NULL when unused. */
void solref_qknorm_rope3d(const uint16_t* x, uint16_t* y, double* yf, int64_t rows, int N, int D,
                          int T, int Hl, int Wl, int dt, int dh, int dw, double base, int rope,
                          const double* gamma, double eps, int contract) {
  double* buf = (double*)malloc(sizeof(double) * (size_t)D);
  for (int64_t r = 0; r < rows; ++r) {
    int64_t n = r % N;
    rotate_row(x + r * D, buf, n, N, D, T, Hl, Wl, dt, dh, dw, base, rope, 0, gamma, eps);
    for (int d = 0; d < D; ++d) {
      if (contract) y[r * D + d] = double_to_bf16(buf[d]);
      else yf[r * D + d] = buf[d];
    }
  }
  free(buf);
}

/* ------------------------------------------------------------------ attention */

/* Where the rows of one side (queries, or keys and values) sit in their
 * sequence, and what is done to them before the products. */
typedef struct {
  int N, T, Hl, Wl;       /* sequence length and latent grid (prefix = N - T*Hl*Wl) */
  int rope;               /* rotate (3D rotary embedding) */
  const double* gamma;    /* RMS-normalise with these D weights first, or NULL */
} side_t;

typedef struct {
  /* one (b,h) slab */
  const uint16_t* q;      /* [Nq][D] */
  const double* khat;     /* [Nkv][D] prepared keys */
  const double* vd;       /* [Nkv][D] */
  side_t qs;
  int Nkv, D, dt, dh, dw, contract;
  double base, eps;
  const uint8_t* bmask;   /* block mask of the slab [nqb][nkb], or NULL (dense) */
  int qblk, kblk, nkb;    /* query / key block sizes, key blocks per slab */
  const int64_t* qrows;   /* query indices within the slab */
  float* out;             /* [nq][D] */
  int64_t nq;
  int64_t next;           /* shared work counter */
  pthread_mutex_t lock;
} slab_job;

static void attend_one(slab_job* J, int64_t idx, double* s, double* qhat, double* acc) {
  const int Nkv = J->Nkv, D = J->D;
  int64_t i = J->qrows[idx];
  rotate_row(J->q + i * D, qhat, i, J->qs.N, D, J->qs.T, J->qs.Hl, J->qs.Wl, J->dt, J->dh, J->dw,
             J->base, J->qs.rope, J->contract, J->qs.gamma, J->eps);
  const double scale = 1.0 / sqrt((double)D);
  /* keys this query may attend to: all, or those of its block's kept key blocks */
  const uint8_t* keep = J->bmask ? J->bmask + (i / J->qblk) * (int64_t)J->nkb : NULL;
  /* pass 1: logits and their maximum */
  double m = -INFINITY;
  for (int j = 0; j < Nkv; ++j) {
    const double* kj = J->khat + (int64_t)j * D;
    double dot = 0.0;
    for (int d = 0; d < D; ++d) dot += qhat[d] * kj[d];
    s[j] = dot * scale;
    if (keep && !keep[j / J->kblk]) s[j] = -INFINITY;
    if (s[j] > m) m = s[j];
  }
  /* pass 2: exponentials, normaliser, weighted sum of values */
  double l = 0.0;
  for (int d = 0; d < D; ++d) acc[d] = 0.0;
  for (int j = 0; j < Nkv; ++j) {
    if (s[j] == -INFINITY) continue; /* a key outside the kept blocks */
    double p = exp(s[j] - m);
    l += p;
    const double* vj = J->vd + (int64_t)j * D;
    for (int d = 0; d < D; ++d) acc[d] += p * vj[d];
  }
  for (int d = 0; d < D; ++d) J->out[idx * D + d] = (float)(acc[d] / l);
}

/* Rotation of one slab's keys (and widening of its values), split over threads. */
typedef struct {
  const uint16_t* ks;
  const uint16_t* vs;
  double* khat;
  double* vd;
  side_t kside;
  int D, dt, dh, dw, contract;
  double base, eps;
  int64_t next;
  pthread_mutex_t lock;
} keys_job;

static void* keys_worker(void* arg) {
  keys_job* J = (keys_job*)arg;
  const int D = J->D, N = J->kside.N;
  for (;;) {
    pthread_mutex_lock(&J->lock);
    int64_t j0 = J->next;
    J->next += 256;
    pthread_mutex_unlock(&J->lock);
    if (j0 >= N) break;
    int64_t j1 = j0 + 256 < N ? j0 + 256 : N;
    for (int64_t j = j0; j < j1; ++j) {
      rotate_row(J->ks + j * D, J->khat + j * D, j, N, D, J->kside.T, J->kside.Hl, J->kside.Wl,
                 J->dt, J->dh, J->dw, J->base, J->kside.rope, J->contract, J->kside.gamma, J->eps);
      for (int d = 0; d < D; ++d) J->vd[j * D + d] = bf16_to_double(J->vs[j * D + d]);
    }
  }
  return NULL;
}

static void* slab_worker(void* arg) {
  slab_job* J = (slab_job*)arg;
  double* s = (double*)malloc(sizeof(double) * (size_t)J->Nkv);
  double* qhat = (double*)malloc(sizeof(double) * (size_t)J->D);
  double* acc = (double*)malloc(sizeof(double) * (size_t)J->D);
  for (;;) {
    pthread_mutex_lock(&J->lock);
    int64_t idx = J->next++;
    pthread_mutex_unlock(&J->lock);
    if (idx >= J->nq) break;
    attend_one(J, idx, s, qhat, acc);
  }
  free(s);
  free(qhat);
  free(acc);
  return NULL;
}

int solref_num_threads(void) {
  cpu_set_t set;
  if (sched_getaffinity(0, sizeof set, &set) == 0) return CPU_COUNT(&set);
  return 1;
}

static int bad_side(const side_t* s, int D, int dt, int dh, int dw) {
  if (s->N < 1) return 1;
  if (s->rope && ((int64_t)s->T * s->Hl * s->Wl > s->N || dt + dh + dw > D || s->T < 0 ||
                  s->Hl < 0 || s->Wl < 0))
    return 1;
  return 0;
}

/*
 * Attention output for selected query rows, queries and keys of any lengths.
 *   q          : bf16 bits [B][H][Nq][D];  k, v : bf16 bits [B][H][Nkv][D]
 *   q side     : grid Tq x Hlq x Wlq of the Nq queries, rotated if rope_q,
 *                RMS-normalised first with q_gamma[D] if it is not NULL
 *   k side     : likewise for the Nkv keys (grid Tk x Hlk x Wlk, rope_k,
 *                k_gamma); values are never changed
 *   eps        : added under the root of every RMS normalisation
 *   rows       : global row ids r = (b*H + h)*Nq + i, grouped by (b,h) in any order
 *   out        : float [nrows][D], row k is the output for rows[k]
 *   nthreads   : <= 0 means every CPU in the affinity mask
 * Returns 0, or -1 on bad arguments / allocation failure.
 */
static int attn_rows_impl(const uint16_t* q, const uint16_t* k, const uint16_t* v, int B, int H,
                          int Nq, int Nkv, int D, int Tq, int Hlq, int Wlq, int Tk, int Hlk, int Wlk,
                          int dt, int dh, int dw, double base, int rope_q, int rope_k, int contract,
                          const double* q_gamma, const double* k_gamma, double eps,
                          const uint8_t* bmask, int qblk, int kblk,
                          const int64_t* rows, int64_t nrows, float* out, int nthreads) {
  const side_t qs = {Nq, Tq, Hlq, Wlq, rope_q, q_gamma};
  const side_t ks = {Nkv, Tk, Hlk, Wlk, rope_k, k_gamma};
  if (B < 1 || H < 1 || D < 2 || !q || !k || !v || !out || (nrows > 0 && !rows)) return -1;
  if (bmask && (qblk < 1 || kblk < 1)) return -1;
  const int nqb = bmask ? (Nq + qblk - 1) / qblk : 0;
  const int nkb = bmask ? (Nkv + kblk - 1) / kblk : 0;
  if (bad_side(&qs, D, dt, dh, dw) || bad_side(&ks, D, dt, dh, dw) || !(eps >= 0.0)) return -1;
  if (nthreads <= 0) nthreads = solref_num_threads();
  const int64_t qslab = (int64_t)Nq * D, kslab = (int64_t)Nkv * D;
  int64_t* qrows = (int64_t*)malloc(sizeof(int64_t) * (size_t)(nrows > 0 ? nrows : 1));
  int64_t* where = (int64_t*)malloc(sizeof(int64_t) * (size_t)(nrows > 0 ? nrows : 1));
  float* obuf = (float*)malloc(sizeof(float) * (size_t)(nrows > 0 ? nrows : 1) * D);
  double* khat = (double*)malloc(sizeof(double) * (size_t)kslab);
  double* vd = (double*)malloc(sizeof(double) * (size_t)kslab);
  pthread_t* th = (pthread_t*)malloc(sizeof(pthread_t) * (size_t)nthreads);
  if (!qrows || !where || !obuf || !khat || !vd || !th) {
    free(qrows); free(where); free(obuf); free(khat); free(vd); free(th);
    return -1;
  }
  for (int64_t r = 0; r < nrows; ++r) {
    if (rows[r] < 0 || rows[r] >= (int64_t)B * H * Nq) {
      free(qrows); free(where); free(obuf); free(khat); free(vd); free(th);
      return -1;
    }
  }
  for (int64_t bh = 0; bh < (int64_t)B * H; ++bh) {
    /* collect the requested rows of this slab */
    int64_t nq = 0;
    for (int64_t r = 0; r < nrows; ++r) {
      if (rows[r] / Nq == bh) {
        qrows[nq] = rows[r] % Nq;
        where[nq] = r;
        ++nq;
      }
    }
    if (nq == 0) continue;
    keys_job K;
    K.ks = k + bh * kslab;
    K.vs = v + bh * kslab;
    K.khat = khat;
    K.vd = vd;
    K.kside = ks;
    K.D = D; K.dt = dt; K.dh = dh; K.dw = dw; K.base = base; K.eps = eps;
    K.contract = contract;
    K.next = 0;
    pthread_mutex_init(&K.lock, NULL);
    for (int t = 0; t < nthreads; ++t) pthread_create(&th[t], NULL, keys_worker, &K);
    for (int t = 0; t < nthreads; ++t) pthread_join(th[t], NULL);
    pthread_mutex_destroy(&K.lock);
    slab_job J;
    J.q = q + bh * qslab;
    J.khat = khat;
    J.vd = vd;
    J.qs = qs;
    J.Nkv = Nkv; J.D = D; J.dt = dt; J.dh = dh; J.dw = dw; J.base = base; J.eps = eps;
    J.bmask = bmask ? bmask + bh * (int64_t)nqb * nkb : NULL;
    J.qblk = qblk; J.kblk = kblk; J.nkb = nkb;
    J.contract = contract;
    J.qrows = qrows;
    J.out = obuf;
    J.nq = nq;
    J.next = 0;
    pthread_mutex_init(&J.lock, NULL);
    int nt = nthreads < nq ? nthreads : (int)nq;
    for (int t = 0; t < nt; ++t) pthread_create(&th[t], NULL, slab_worker, &J);
    for (int t = 0; t < nt; ++t) pthread_join(th[t], NULL);
    pthread_mutex_destroy(&J.lock);
    for (int64_t r = 0; r < nq; ++r) memcpy(out + where[r] * D, obuf + r * D, sizeof(float) * D);
  }
  free(qrows); free(where); free(obuf); free(khat); free(vd); free(th);
  return 0;
}

int solref_attn_rows_ex(const uint16_t* q, const uint16_t* k, const uint16_t* v, int B, int H,
                        int Nq, int Nkv, int D, int Tq, int Hlq, int Wlq, int Tk, int Hlk, int Wlk,
                        int dt, int dh, int dw, double base, int rope_q, int rope_k, int contract,
                        const double* q_gamma, const double* k_gamma, double eps,
                        const int64_t* rows, int64_t nrows, float* out, int nthreads) {
  return attn_rows_impl(q, k, v, B, H, Nq, Nkv, D, Tq, Hlq, Wlq, Tk, Hlk, Wlk, dt, dh, dw, base,
                        rope_q, rope_k, contract, q_gamma, k_gamma, eps, NULL, 0, 0, rows, nrows,
                        out, nthreads);
}

/* Block-sparse attention: as solref_attn_rows_ex, but query i of slab bh
 * attends only to the keys of the key blocks J (kblk keys each, from key 0)
 * with bmask[bh][i / qblk][J] != 0 (bmask: [B*H][ceil(Nq/qblk)][ceil(Nkv/kblk)]);
 * the softmax runs over those keys alone. */
int solref_attn_rows_sparse(const uint16_t* q, const uint16_t* k, const uint16_t* v, int B, int H,
                            int Nq, int Nkv, int D, int Tq, int Hlq, int Wlq, int Tk, int Hlk,
                            int Wlk, int dt, int dh, int dw, double base, int rope_q, int rope_k,
                            int contract, const double* q_gamma, const double* k_gamma, double eps,
                            const uint8_t* bmask, int qblk, int kblk, const int64_t* rows,
                            int64_t nrows, float* out, int nthreads) {
  if (!bmask) return -1;
  return attn_rows_impl(q, k, v, B, H, Nq, Nkv, D, Tq, Hlq, Wlq, Tk, Hlk, Wlk, dt, dh, dw, base,
                        rope_q, rope_k, contract, q_gamma, k_gamma, eps, bmask, qblk, kblk, rows,
                        nrows, out, nthreads);
}

/*
 * Block routing of the block-sparse attention (Sec. 3.4, "Per-step dynamic
 * sparsity" and "Safety rails and the exact prefix KV sink"), for the
 * self-attention of B*H slabs of N tokens (grid T x Hl x Wl; the first
 * Nt = N - T*Hl*Wl tokens are the prefix).  Query blocks of qblk rows and key
 * blocks of kblk keys, both counted from token 0.  With q^, k^ the rows as they
 * enter the products (normalised if a gamma is given, rotated if rope, rounded
 * to bf16 if contract):
 *   qbar_I = mean of q^_i over the rows of block I, kbar_J likewise for keys;
 *   s_IJ  = <qbar_I, kbar_J> / sqrt(D)          (the block-level score);
 *   mu_I, sigma_I = mean and population standard deviation of s_IJ over all J;
 *   key block J is kept for query block I iff s_IJ > mu_I + tau sigma_I, or J
 *   holds a prefix key (the exact prefix sink), or J is the first block with
 *   the largest s_IJ (so no block attends to nothing); a query block that
 *   holds a prefix row keeps every key block (prefix queries attend densely).
 * Outputs (each may be NULL): mask [B*H][nqb][nkb] (1 = kept), scores s_IJ
 * [B*H][nqb][nkb] and thresholds mu_I + tau sigma_I [B*H][nqb].
 */
int solref_sparse_route(const uint16_t* q, const uint16_t* k, int BH, int N, int D, int T, int Hl,
                        int Wl, int dt, int dh, int dw, double base, int rope, int contract,
                        const double* q_gamma, const double* k_gamma, double eps, int qblk,
                        int kblk, double tau, uint8_t* mask, double* scores, double* thr) {
  if (BH < 1 || N < 1 || D < 2 || qblk < 1 || kblk < 1 || !q || !k) return -1;
  if ((int64_t)T * Hl * Wl > N || T < 0 || Hl < 0 || Wl < 0) return -1;
  const int64_t nt = (int64_t)N - (int64_t)T * Hl * Wl;
  const int nqb = (N + qblk - 1) / qblk, nkb = (N + kblk - 1) / kblk;
  double* qbar = (double*)calloc((size_t)nqb * D, sizeof(double));
  double* kbar = (double*)calloc((size_t)nkb * D, sizeof(double));
  double* row = (double*)malloc(sizeof(double) * (size_t)D);
  double* s = (double*)malloc(sizeof(double) * (size_t)nkb);
  if (!qbar || !kbar || !row || !s) {
    free(qbar); free(kbar); free(row); free(s);
    return -1;
  }
  const double scale = 1.0 / sqrt((double)D);
  for (int64_t bh = 0; bh < BH; ++bh) {
    const uint16_t* qs = q + bh * (int64_t)N * D;
    const uint16_t* ks = k + bh * (int64_t)N * D;
    memset(qbar, 0, sizeof(double) * (size_t)nqb * D);
    memset(kbar, 0, sizeof(double) * (size_t)nkb * D);
    for (int64_t n = 0; n < N; ++n) {
      rotate_row(qs + n * D, row, n, N, D, T, Hl, Wl, dt, dh, dw, base, rope, contract, q_gamma, eps);
      for (int d = 0; d < D; ++d) qbar[(n / qblk) * D + d] += row[d];
      rotate_row(ks + n * D, row, n, N, D, T, Hl, Wl, dt, dh, dw, base, rope, contract, k_gamma, eps);
      for (int d = 0; d < D; ++d) kbar[(n / kblk) * D + d] += row[d];
    }
    for (int I = 0; I < nqb; ++I) {
      const int64_t rows = (I + 1) * (int64_t)qblk <= N ? qblk : N - (int64_t)I * qblk;
      for (int d = 0; d < D; ++d) qbar[I * D + d] /= (double)rows;
    }
    for (int J = 0; J < nkb; ++J) {
      const int64_t keys = (J + 1) * (int64_t)kblk <= N ? kblk : N - (int64_t)J * kblk;
      for (int d = 0; d < D; ++d) kbar[J * D + d] /= (double)keys;
    }
    for (int I = 0; I < nqb; ++I) {
      double mu = 0.0, var = 0.0;
      int best = 0;
      for (int J = 0; J < nkb; ++J) {
        double dot = 0.0;
        for (int d = 0; d < D; ++d) dot += qbar[I * D + d] * kbar[J * D + d];
        s[J] = dot * scale;
        mu += s[J];
        if (s[J] > s[best]) best = J;
      }
      mu /= (double)nkb;
      for (int J = 0; J < nkb; ++J) var += (s[J] - mu) * (s[J] - mu);
      const double t = mu + tau * sqrt(var / (double)nkb);
      const int dense = (int64_t)I * qblk < nt; /* the block holds a prefix row */
      const int64_t o = (bh * nqb + I) * (int64_t)nkb;
      for (int J = 0; J < nkb; ++J) {
        const int sink = (int64_t)J * kblk < nt; /* the block holds a prefix key */
        if (mask) mask[o + J] = (uint8_t)(dense || sink || J == best || s[J] > t);
        if (scores) scores[o + J] = s[J];
      }
      if (thr) thr[bh * nqb + I] = t;
    }
  }
  free(qbar); free(kbar); free(row); free(s);
  return 0;
}

/* Self-attention of one sequence (queries and keys the same N tokens, one
 * grid, no normalisation): solref_attn_rows_ex with both sides alike. */
int solref_attn_rows(const uint16_t* q, const uint16_t* k, const uint16_t* v,
                     int B, int H, int N, int D, int T, int Hl, int Wl,
                     int dt, int dh, int dw, double base, int use_rope, int contract,
                     const int64_t* rows, int64_t nrows, float* out, int nthreads) {
  return solref_attn_rows_ex(q, k, v, B, H, N, N, D, T, Hl, Wl, T, Hl, Wl, dt, dh, dw, base,
                             use_rope, use_rope, contract, NULL, NULL, 0.0, rows, nrows, out,
                             nthreads);
}

/* ------------------------------------------------- block-INT8 QKV records */

/*
 * The wire record of the quantized QKV exchange (Sec. 3.2, "Quantized
 * communication"): one record per (token, head), 400 bytes -- 384 bytes of
 * int8 codes, twelve scale codes (one per group of 32 values) and four zero
 * bytes.  Readings where the paper gives only the sizes:
 *   bytes   0..127  q codes, 128..255 k codes, 256..383 v codes (two's
 *                   complement; dim d of a part at byte d of that part);
 *   bytes 384..395  scale code of part p (0 q, 1 k, 2 v), dims [32g, 32g+32)
 *                   at byte 384 + 4p + g;
 *   bytes 396..399  zero.
 * Records are token-major, (b, n, h) at byte ((b*N + n)*H + h)*400: the flat
 * (tokens, heads, record) layout the exchange delivers.
 *
 * UE5M3 scale codes (reading): unsigned, 5 exponent bits of bias 15, 3
 * mantissa bits; exponent 0 is subnormal (m * 2^-17), exponent 31 is not
 * finite (m = 0 infinity, else NaN).  The finite positive codes 0x01..0xF7
 * span 2^-17 .. 61440.
 *
 * Encoding (reading): a group's scale is the smallest finite positive code
 * value s with 127 s >= max |x| (no value needs a code beyond +-127; a zero
 * group takes 0x01, a group too large for any code 0xF7); each value's code
 * is x / s rounded to the nearest integer, ties to even, clamped to
 * [-127, 127].  The inputs are the bf16 q, k and v as attention consumes them
 * (q and k normalised and rotated), finite.
 * Decoding: code * s rounded once to bf16 (RNE), the rounding point at which
 * a bf16 consumer receives them.
 */
#define REC_BYTES 400
#define REC_SCALES 384

static double ue5m3_value(uint8_t c) {
  int e = c >> 3, m = c & 7;
  if (e == 31) return m == 0 ? INFINITY : NAN;
  if (e == 0) return ldexp((double)m, -17);
  return ldexp(8.0 + m, e - 18); /* (1 + m/8) 2^(e-15) */
}

/* The first code c in 1..0xF7 with 127 value(c) >= amax (0xF7 if none):
 * value() increases with the code, so the codes that pass form a suffix of
 * 1..0xF7 and halving the interval finds its start. */
static uint8_t ue5m3_scale_for(double amax) {
  int first = 1, past = 0xF7; /* the answer lies in [first, past] */
  while (first < past) {
    int mid = (first + past) / 2;
    if (127.0 * ue5m3_value((uint8_t)mid) >= amax) past = mid;
    else first = mid + 1;
  }
  return (uint8_t)first;
}

static int8_t int8_code(double x, double s) {
  double y = x / s;
  double fl = floor(y);
  double rem = y - fl;
  if (rem > 0.5 || (rem == 0.5 && fmod(fl, 2.0) != 0.0)) fl += 1.0;
  if (fl > 127.0) fl = 127.0;
  if (fl < -127.0) fl = -127.0;
  return (int8_t)fl;
}

/* q, k, v: bf16 bits [B][H][N][D], D = 128; rec: [B][N][H][400]. */
int solref_encode_qkv(const uint16_t* q, const uint16_t* k, const uint16_t* v, int B, int H,
                      int N, int D, uint8_t* rec) {
  if (D != 128 || B < 1 || H < 1 || N < 1 || !q || !k || !v || !rec) return -1;
  const uint16_t* part[3] = {q, k, v};
  for (int b = 0; b < B; ++b)
    for (int n = 0; n < N; ++n)
      for (int h = 0; h < H; ++h) {
        uint8_t* r = rec + (((int64_t)b * N + n) * H + h) * REC_BYTES;
        for (int p = 0; p < 3; ++p) {
          const uint16_t* x = part[p] + (((int64_t)b * H + h) * N + n) * D;
          for (int g = 0; g < 4; ++g) {
            double amax = 0.0;
            for (int d = 32 * g; d < 32 * g + 32; ++d) amax = fmax(amax, fabs(bf16_to_double(x[d])));
            const uint8_t sc = ue5m3_scale_for(amax);
            const double s = ue5m3_value(sc);
            r[REC_SCALES + 4 * p + g] = sc;
            for (int d = 32 * g; d < 32 * g + 32; ++d)
              r[128 * p + d] = (uint8_t)int8_code(bf16_to_double(x[d]), s);
          }
        }
        for (int i = REC_SCALES + 12; i < REC_BYTES; ++i) r[i] = 0;
      }
  return 0;
}

/* rec: [B][N][H][400] -> q, k, v bf16 bits [B][H][N][D], D = 128. */
int solref_decode_qkv(const uint8_t* rec, int B, int H, int N, int D, uint16_t* q, uint16_t* k,
                      uint16_t* v) {
  if (D != 128 || B < 1 || H < 1 || N < 1 || !rec || !q || !k || !v) return -1;
  uint16_t* part[3] = {q, k, v};
  for (int b = 0; b < B; ++b)
    for (int n = 0; n < N; ++n)
      for (int h = 0; h < H; ++h) {
        const uint8_t* r = rec + (((int64_t)b * N + n) * H + h) * REC_BYTES;
        for (int p = 0; p < 3; ++p) {
          uint16_t* x = part[p] + (((int64_t)b * H + h) * N + n) * D;
          for (int d = 0; d < D; ++d) {
            const double s = ue5m3_value(r[REC_SCALES + 4 * p + d / 32]);
            x[d] = double_to_bf16((double)(int8_t)r[128 * p + d] * s);
          }
        }
      }
  return 0;
}

/*
 * Block-INT8 output records (Sec. 3.2, "Quantized communication": the
 * attention output's block-INT8 wire format, 128 value bytes and four scale
 * codes, padded from 132 to 144 bytes).  Reading: bytes 0..127 the int8
 * codes of the 128 output dims, bytes 128..131 the UE5M3 scale codes of dims
 * [32g, 32g + 32), bytes 132..143 zero; the codes and scales follow the QKV
 * records' rule, applied to the exact (double) attention output.
 * x: double [rows][128]; rec: [rows][144].
 */
#define OUT_REC_BYTES 144
void solref_encode_out_records(const double* x, int64_t rows, uint8_t* rec) {
  for (int64_t r = 0; r < rows; ++r) {
    const double* xr = x + r * 128;
    uint8_t* o = rec + r * OUT_REC_BYTES;
    for (int g = 0; g < 4; ++g) {
      double amax = 0.0;
      for (int d = 32 * g; d < 32 * g + 32; ++d) amax = fmax(amax, fabs(xr[d]));
      const uint8_t sc = ue5m3_scale_for(amax);
      const double s = ue5m3_value(sc);
      o[128 + g] = sc;
      for (int d = 32 * g; d < 32 * g + 32; ++d) o[d] = (uint8_t)int8_code(xr[d], s);
    }
    for (int i = 132; i < OUT_REC_BYTES; ++i) o[i] = 0;
  }
}
