/*
 * jl_oracle.c -- fp64 CPU oracle for Jet-Long bifocal-RoPE attention.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path links, loads or
 * calls this file: only the test suite, the smoke check and the benchmark's
 * CPU-baseline leg do.  It shares no code, header, table or constant with the
 * HIP implementation.
 *
 * It computes what Jet-Long (arXiv 2607.07740) defines, written for a reader
 * to check by eye against the paper, slowly and in double precision:
 *
 *   - group size  G = max(1, ceil(L / w_pretrained))           Sec. 3.1, Eq. (2)
 *   - remote map  f(x) = floor(x / G)                            Sec. 3.1, Eq. (3)
 *   - two-window score: base RoPE if q - k <= w0, else RoPE at
 *     f(q), f(k)                                                 Sec. 3, Eq. (1)
 *   - prefill output as three separate softmax windows
 *       A: keys [q - w0, q], base rotation
 *       B: keys [0, q],      remote rotation
 *       C: keys [q - w0, q], remote rotation
 *     each returning (O_X, lse_X), merged by inclusion-exclusion  Sec. 3.3, Eq. (7)
 *   - decode: the same row at q = kv_len - 1 with G taken from
 *     L = kv_len (the cache holds raw keys, rotated on the fly)  Sec. 3.2, Eqs. (4)-(6)
 *   - the ablated remote map of Sec. 4.5, Table 6: remote keys keep their
 *     positions and are rotated with YaRN-style rescaled frequencies instead
 *     of being aliased to f(x)
 *
 * RoPE convention (the paper does not print it; rotate-half pairing of the
 * Qwen3 family is assumed): for i < d/2 with omega_i = theta^(-2i/d),
 *   y_i       = x_i cos(p omega_i) - x_{i+d/2} sin(p omega_i)
 *   y_{i+d/2} = x_{i+d/2} cos(p omega_i) + x_i sin(p omega_i).
 * Every position is rotated explicitly (the direct form R(f(k)) x_k, not the
 * correction form R(Delta k) R(k) x_k; the two agree by R_a R_b = R_{a+b},
 * Sec. 3.2).  Softmax scale 1/sqrt(d); positions are 0-based; GQA maps query
 * head h to kv head h / (Hq / Hkv).
 *
 * Inputs are bf16 bit patterns (uint16), converted exactly to double.
 * Parity pins for every function here live in the CPU test suite.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define JLO_OK 0
#define JLO_EINVAL 1
#define JLO_ENOMEM 2

static double bf16_to_double(uint16_t bits) {
  uint32_t u = (uint32_t)bits << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return (double)f;
}

/* Sec. 3.1, Eq. (2): the smallest integer G >= 1 with ceil(L / G) <= w. */
int64_t jlo_group_size(int64_t L, int64_t w_pretrained) {
  if (L < 1 || w_pretrained < 1) return -1;
  int64_t G = L / w_pretrained;
  if (G * w_pretrained < L) G += 1; /* ceiling */
  if (G < 1) G = 1;
  return G;
}

/* Sec. 3.1, Eq. (3): floor(x / G) for x >= 0, G >= 1. */
int64_t jlo_remote_position(int64_t x, int64_t G) {
  if (x < 0 || G < 1) return -1;
  return x / G;
}

/* Sec. 3.2, Eq. (5): Delta(x) = f(x) - x. */
int64_t jlo_position_offset(int64_t x, int64_t G) {
  int64_t f = jlo_remote_position(x, G);
  if (f < 0) return 1; /* invalid: a valid offset is never positive */
  return f - x;
}

/* Explicit RoPE rotation of one d-vector to position pos (may be negative:
 * a rotation by a negative angle).  Angles p * omega_i in fp64. */
void jlo_rope_rotate(const double* x, int d, double pos, double theta, double* y) {
  int half = d / 2;
  for (int i = 0; i < half; ++i) {
    double omega = pow(theta, -2.0 * (double)i / (double)d);
    double ang = pos * omega;
    double c = cos(ang), s = sin(ang);
    double a = x[i], b = x[i + half];
    y[i] = a * c - b * s;
    y[i + half] = b * c + a * s;
  }
}

/* The same rotation with explicit per-pair angular frequencies omega[i]. */
void jlo_rope_rotate_freqs(const double* x, int d, double pos, const double* omega, double* y) {
  int half = d / 2;
  for (int i = 0; i < half; ++i) {
    double ang = pos * omega[i];
    double c = cos(ang), s = sin(ang);
    double a = x[i], b = x[i + half];
    y[i] = a * c - b * s;
    y[i + half] = b * c + a * s;
  }
}

/*
 * Frequencies of the frequency-interpolation remote map (the ablation of
 * Sec. 4.5, Table 6, that keeps positions and rescales frequencies, in the
 * style of YaRN).  The
 * continuous factor is the one Sec. 3.1 names for such methods,
 * s = max(1, L / w_pretrained).  Per pair i, following YaRN's per-dimension
 * rule: wavelength lambda_i = 2 pi / omega_i, r_i = w_pretrained / lambda_i
 * (turns completed over the pretraining window), ramp
 *   gamma = 0 if r_i < alpha,  1 if r_i > beta,  (r_i - alpha) / (beta - alpha) else,
 * and omega'_i = (1 - gamma) omega_i / s + gamma omega_i: pairs that turn
 * many times inside the window keep their frequency, slow pairs are divided
 * by s.  No attention temperature (only the rotation is replaced).
 * omega_out: d/2 values.
 */
void jlo_yarn_frequencies(int d, double theta, double L, double w_pretrained, double alpha,
                          double beta, double* omega_out) {
  double s = L / w_pretrained;
  if (s < 1.0) s = 1.0;
  int half = d / 2;
  for (int i = 0; i < half; ++i) {
    double omega = pow(theta, -2.0 * (double)i / (double)d);
    double lambda = 2.0 * acos(-1.0) / omega;
    double r = w_pretrained / lambda;
    double gamma;
    if (r < alpha)
      gamma = 0.0;
    else if (r > beta)
      gamma = 1.0;
    else
      gamma = (r - alpha) / (beta - alpha);
    omega_out[i] = (1.0 - gamma) * omega / s + gamma * omega;
  }
}

/* One softmax "call" over a key set: returns O (d values) and the natural-log
 * LSE of the scores.  scores[j] are already divided by sqrt(d). */
static double softmax_call(const double* scores, const double* const* vals, int64_t n, int d,
                           double* out) {
  double m = -INFINITY;
  for (int64_t j = 0; j < n; ++j)
    if (scores[j] > m) m = scores[j];
  double z = 0.0;
  for (int c = 0; c < d; ++c) out[c] = 0.0;
  for (int64_t j = 0; j < n; ++j) {
    double w = exp(scores[j] - m);
    z += w;
    for (int c = 0; c < d; ++c) out[c] += w * vals[j][c];
  }
  for (int c = 0; c < d; ++c) out[c] /= z;
  return m + log(z);
}

static double dot(const double* a, const double* b, int d) {
  double s = 0.0;
  for (int c = 0; c < d; ++c) s += a[c] * b[c];
  return s;
}

/*
 * Per (b, kv-head) rotated keys: kb[k] = R(k) x_k and kr[k] = R(f(k)) x_k for
 * k < n_keys (or, with remote frequencies romega, kr[k] = R'(k) x_k at the
 * unchanged position), plus raw values, all in fp64.  key_stride is the
 * distance in elements between consecutive positions of one head.
 */
typedef struct {
  int64_t n;
  int d;
  double* kb;
  double* kr;
  double* v;
} keyset_t;

static int keyset_build(keyset_t* ks, const uint16_t* k, const uint16_t* v, int64_t n, int d,
                        int64_t key_stride, int64_t G, double theta, int want_remote,
                        const double* romega) {
  ks->n = n;
  ks->d = d;
  ks->kb = (double*)malloc(sizeof(double) * (size_t)(n * d));
  ks->kr = want_remote ? (double*)malloc(sizeof(double) * (size_t)(n * d)) : NULL;
  ks->v = (double*)malloc(sizeof(double) * (size_t)(n * d));
  if (!ks->kb || !ks->v || (want_remote && !ks->kr)) return JLO_ENOMEM;
  int failed = 0;
#pragma omp parallel
  {
    double* raw = (double*)malloc(sizeof(double) * (size_t)d);
    if (!raw) {
#pragma omp atomic write
      failed = 1;
    }
#pragma omp for schedule(static)
    for (int64_t j = 0; j < n; ++j) {
      if (!raw) continue;
      for (int c = 0; c < d; ++c) raw[c] = bf16_to_double(k[j * key_stride + c]);
      jlo_rope_rotate(raw, d, (double)j, theta, ks->kb + j * d);
      if (want_remote && romega)
        jlo_rope_rotate_freqs(raw, d, (double)j, romega, ks->kr + j * d);
      else if (want_remote)
        jlo_rope_rotate(raw, d, (double)jlo_remote_position(j, G), theta, ks->kr + j * d);
      for (int c = 0; c < d; ++c) ks->v[j * d + c] = bf16_to_double(v[j * key_stride + c]);
    }
    free(raw);
  }
  return failed ? JLO_ENOMEM : JLO_OK;
}

static void keyset_free(keyset_t* ks) {
  free(ks->kb);
  free(ks->kr);
  free(ks->v);
}

/*
 * One bifocal output row, Sec. 3.3: windows A, B, C computed separately, then
 * merged by Eq. (7) with M = max(lse_A, lse_B, lse_C), W_X = exp(lse_X - M).
 * xq: raw query (fp64, d); qpos: its 0-based position; G: the call's group
 * size; w0: local window; romega: NULL for the aliasing map f, else the
 * remote frequencies (the query keeps its position).  Writes out[d] and
 * returns the merged LSE.
 */
static double bifocal_row(const double* xq, int64_t qpos, int64_t G, int64_t w0, double theta,
                          const keyset_t* ks, const double* romega, double* out) {
  int d = ks->d;
  double scale = 1.0 / sqrt((double)d);
  double* qb = (double*)malloc(sizeof(double) * (size_t)d);
  double* qr = (double*)malloc(sizeof(double) * (size_t)d);
  double* oa = (double*)malloc(sizeof(double) * (size_t)d);
  double* ob = (double*)malloc(sizeof(double) * (size_t)d);
  double* oc = (double*)malloc(sizeof(double) * (size_t)d);
  int64_t nb = qpos + 1;
  double* s = (double*)malloc(sizeof(double) * (size_t)nb);
  const double** vv = (const double**)malloc(sizeof(double*) * (size_t)nb);
  jlo_rope_rotate(xq, d, (double)qpos, theta, qb);
  if (romega)
    jlo_rope_rotate_freqs(xq, d, (double)qpos, romega, qr);
  else
    jlo_rope_rotate(xq, d, (double)jlo_remote_position(qpos, G), theta, qr);

  int64_t lo = qpos - w0;
  if (lo < 0) lo = 0;
  int64_t na = qpos - lo + 1;

  /* A: sliding window (local w0), base queries and keys. */
  for (int64_t j = 0; j < na; ++j) {
    s[j] = dot(qb, ks->kb + (lo + j) * d, d) * scale;
    vv[j] = ks->v + (lo + j) * d;
  }
  double la = softmax_call(s, vv, na, d, oa);

  /* B: full causal attention, remote queries and keys. */
  for (int64_t j = 0; j < nb; ++j) {
    s[j] = dot(qr, ks->kr + j * d, d) * scale;
    vv[j] = ks->v + j * d;
  }
  double lb = softmax_call(s, vv, nb, d, ob);

  /* C: sliding window (local w0), remote queries and keys. */
  for (int64_t j = 0; j < na; ++j) {
    s[j] = dot(qr, ks->kr + (lo + j) * d, d) * scale;
    vv[j] = ks->v + (lo + j) * d;
  }
  double lc = softmax_call(s, vv, na, d, oc);

  /* Eq. (7). */
  double M = la;
  if (lb > M) M = lb;
  if (lc > M) M = lc;
  double wa = exp(la - M), wb = exp(lb - M), wc = exp(lc - M);
  double den = wa + wb - wc;
  for (int c = 0; c < d; ++c) out[c] = (wa * oa[c] + wb * ob[c] - wc * oc[c]) / den;
  double lse = M + log(den);

  free(qb); free(qr); free(oa); free(ob); free(oc); free(s); free(vv);
  return lse;
}

/* Vanilla causal RoPE attention row (the base model; Sec. 3, L <= w_pretrained). */
static double rope_row(const double* xq, int64_t qpos, double theta, const keyset_t* ks,
                       double* out) {
  int d = ks->d;
  double scale = 1.0 / sqrt((double)d);
  double* qb = (double*)malloc(sizeof(double) * (size_t)d);
  int64_t n = qpos + 1;
  double* s = (double*)malloc(sizeof(double) * (size_t)n);
  const double** vv = (const double**)malloc(sizeof(double*) * (size_t)n);
  jlo_rope_rotate(xq, d, (double)qpos, theta, qb);
  for (int64_t j = 0; j < n; ++j) {
    s[j] = dot(qb, ks->kb + j * d, d) * scale;
    vv[j] = ks->v + j * d;
  }
  double lse = softmax_call(s, vv, n, d, out);
  free(qb); free(s); free(vv);
  return lse;
}

static int check_shape(int B, int Hq, int Hkv, int L, int d, double theta) {
  if (B < 1 || Hq < 1 || Hkv < 1 || L < 1 || d < 2 || (d % 2) != 0) return 0;
  if (Hq % Hkv != 0) return 0;
  if (!(theta > 0.0)) return 0;
  return 1;
}

/*
 * Prefill rows.  q: bf16 [B, L, Hq, d]; k, v: bf16 [B, L, Hkv, d].
 * rows: nrows triples (b, h, qpos).  bifocal != 0 selects Jet-Long, else
 * vanilla RoPE attention (w_pretrained and w0 ignored).  remote_map: 0 = the
 * aliasing map f(x) = floor(x / G) of Eq. (3), 1 = frequency interpolation
 * (jlo_yarn_frequencies with alpha = 1, beta = 32).  out: fp64 [nrows, d];
 * lse (nullable): fp64 [nrows], natural log.  G (or s) is one value for the
 * whole call, from the call's L.  Returns the number of threads used (>= 1)
 * on success, or -JLO_EINVAL / -JLO_ENOMEM.
 */
int jlo_prefill_rows_map(const uint16_t* q, const uint16_t* k, const uint16_t* v, int B, int Hq,
                         int Hkv, int L, int d, double theta, int64_t w_pretrained, int64_t w0,
                         int bifocal, int remote_map, const int64_t* rows, int64_t nrows,
                         double* out, double* lse) {
  if (!check_shape(B, Hq, Hkv, L, d, theta)) return -JLO_EINVAL;
  if (bifocal && (w_pretrained < 1 || w0 < 0)) return -JLO_EINVAL;
  if (remote_map != 0 && remote_map != 1) return -JLO_EINVAL;
  double* romega = NULL;
  if (bifocal && remote_map == 1) {
    romega = (double*)malloc(sizeof(double) * (size_t)(d / 2));
    if (!romega) return -JLO_ENOMEM;
    jlo_yarn_frequencies(d, theta, (double)L, (double)w_pretrained, 1.0, 32.0, romega);
  }
  for (int64_t r = 0; r < nrows; ++r) {
    int64_t b = rows[3 * r], h = rows[3 * r + 1], qp = rows[3 * r + 2];
    if (b < 0 || b >= B || h < 0 || h >= Hq || qp < 0 || qp >= L) return -JLO_EINVAL;
  }
  int64_t G = bifocal ? jlo_group_size(L, w_pretrained) : 1;
  int g = Hq / Hkv;
  int status = JLO_OK;
  int threads = 1;
  /* One (b, kv-head) at a time: rotate its keys once, then its rows in parallel. */
  for (int b = 0; b < B && status == JLO_OK; ++b) {
    for (int kvh = 0; kvh < Hkv && status == JLO_OK; ++kvh) {
      int64_t maxq = -1;
      for (int64_t r = 0; r < nrows; ++r)
        if (rows[3 * r] == b && rows[3 * r + 1] / g == kvh && rows[3 * r + 2] > maxq)
          maxq = rows[3 * r + 2];
      if (maxq < 0) continue;
      keyset_t ks;
      int64_t kstride = (int64_t)Hkv * d;
      const uint16_t* kbase = k + ((int64_t)b * L * Hkv + kvh) * d;
      const uint16_t* vbase = v + ((int64_t)b * L * Hkv + kvh) * d;
      if (keyset_build(&ks, kbase, vbase, maxq + 1, d, kstride, G, theta, bifocal, romega) !=
          JLO_OK) {
        keyset_free(&ks);
        status = JLO_ENOMEM;
        break;
      }
#pragma omp parallel
      {
#ifdef _OPENMP
#pragma omp single
        threads = omp_get_num_threads();
#endif
        double* xq = (double*)malloc(sizeof(double) * (size_t)d);
#pragma omp for schedule(dynamic, 1)
        for (int64_t r = 0; r < nrows; ++r) {
          if (rows[3 * r] != b || rows[3 * r + 1] / g != kvh) continue;
          int64_t h = rows[3 * r + 1], qp = rows[3 * r + 2];
          const uint16_t* qsrc = q + (((int64_t)b * L + qp) * Hq + h) * d;
          for (int c = 0; c < d; ++c) xq[c] = bf16_to_double(qsrc[c]);
          double l = bifocal ? bifocal_row(xq, qp, G, w0, theta, &ks, romega, out + r * d)
                             : rope_row(xq, qp, theta, &ks, out + r * d);
          if (lse) lse[r] = l;
        }
        free(xq);
      }
      keyset_free(&ks);
    }
  }
  free(romega);
  return status == JLO_OK ? threads : -status;
}

/* Prefill rows with the aliasing remote map of Eq. (3). */
int jlo_prefill_rows(const uint16_t* q, const uint16_t* k, const uint16_t* v, int B, int Hq,
                     int Hkv, int L, int d, double theta, int64_t w_pretrained, int64_t w0,
                     int bifocal, const int64_t* rows, int64_t nrows, double* out, double* lse) {
  return jlo_prefill_rows_map(q, k, v, B, Hq, Hkv, L, d, theta, w_pretrained, w0, bifocal, 0,
                              rows, nrows, out, lse);
}

/*
 * Decode: one new query per sequence.  q: bf16 [B, Hq, d] raw, at position
 * kv_lens[b] - 1; k_cache, v_cache: bf16 [B, max_len, Hkv, d] raw (pre-RoPE),
 * only the first kv_lens[b] positions are read.  G per sequence from
 * L = kv_lens[b]; so is the frequency map's factor s = max(1, L / w) when
 * remote_map = 1.  out: fp64 [B, Hq, d]; lse nullable fp64 [B, Hq].
 * Returns threads used (>= 1) or a negative status.
 */
int jlo_decode_map(const uint16_t* q, const uint16_t* k_cache, const uint16_t* v_cache,
                   const int32_t* kv_lens, int max_len, int B, int Hq, int Hkv, int d,
                   double theta, int64_t w_pretrained, int64_t w0, int bifocal, int remote_map,
                   double* out, double* lse) {
  if (!check_shape(B, Hq, Hkv, max_len, d, theta)) return -JLO_EINVAL;
  if (bifocal && (w_pretrained < 1 || w0 < 0)) return -JLO_EINVAL;
  if (remote_map != 0 && remote_map != 1) return -JLO_EINVAL;
  for (int b = 0; b < B; ++b)
    if (kv_lens[b] < 1 || kv_lens[b] > max_len) return -JLO_EINVAL;
  int g = Hq / Hkv;
  int threads = 1;
  int status = JLO_OK;
  double* romega = NULL;
  if (bifocal && remote_map == 1) {
    romega = (double*)malloc(sizeof(double) * (size_t)(d / 2));
    if (!romega) return -JLO_ENOMEM;
  }
  for (int b = 0; b < B && status == JLO_OK; ++b) {
    int64_t n = kv_lens[b];
    int64_t G = bifocal ? jlo_group_size(n, w_pretrained) : 1;
    /* the frequency map's factor follows this sequence's length, as G does */
    if (romega) jlo_yarn_frequencies(d, theta, (double)n, (double)w_pretrained, 1.0, 32.0, romega);
    for (int kvh = 0; kvh < Hkv && status == JLO_OK; ++kvh) {
      keyset_t ks;
      int64_t kstride = (int64_t)Hkv * d;
      const uint16_t* kbase = k_cache + ((int64_t)b * max_len * Hkv + kvh) * d;
      const uint16_t* vbase = v_cache + ((int64_t)b * max_len * Hkv + kvh) * d;
      if (keyset_build(&ks, kbase, vbase, n, d, kstride, G, theta, bifocal, romega) != JLO_OK) {
        keyset_free(&ks);
        status = JLO_ENOMEM;
        break;
      }
#pragma omp parallel
      {
#ifdef _OPENMP
#pragma omp single
        threads = omp_get_num_threads();
#endif
        double* xq = (double*)malloc(sizeof(double) * (size_t)d);
#pragma omp for schedule(static)
        for (int j = 0; j < g; ++j) {
          int64_t h = (int64_t)kvh * g + j;
          const uint16_t* qsrc = q + ((int64_t)b * Hq + h) * d;
          for (int c = 0; c < d; ++c) xq[c] = bf16_to_double(qsrc[c]);
          double* o = out + ((int64_t)b * Hq + h) * d;
          double l = bifocal ? bifocal_row(xq, n - 1, G, w0, theta, &ks, romega, o)
                             : rope_row(xq, n - 1, theta, &ks, o);
          if (lse) lse[(int64_t)b * Hq + h] = l;
        }
        free(xq);
      }
      keyset_free(&ks);
    }
  }
  free(romega);
  return status == JLO_OK ? threads : -status;
}

/* Decode with the aliasing remote map of Eq. (3). */
int jlo_decode(const uint16_t* q, const uint16_t* k_cache, const uint16_t* v_cache,
               const int32_t* kv_lens, int max_len, int B, int Hq, int Hkv, int d, double theta,
               int64_t w_pretrained, int64_t w0, int bifocal, double* out, double* lse) {
  return jlo_decode_map(q, k_cache, v_cache, kv_lens, max_len, B, Hq, Hkv, d, theta,
                        w_pretrained, w0, bifocal, 0, out, lse);
}

/*
 * The three window states of Sec. 3.3 for one prefill row, exposed so the
 * merge itself can be pinned: o3 = [O_A | O_B | O_C] (3*d), lse3 = [lA, lB, lC].
 */
int jlo_window_states(const uint16_t* q, const uint16_t* k, const uint16_t* v, int B, int Hq,
                      int Hkv, int L, int d, double theta, int64_t w_pretrained, int64_t w0,
                      int64_t b, int64_t h, int64_t qpos, double* o3, double* lse3) {
  if (!check_shape(B, Hq, Hkv, L, d, theta) || w_pretrained < 1 || w0 < 0) return -JLO_EINVAL;
  if (b < 0 || b >= B || h < 0 || h >= Hq || qpos < 0 || qpos >= L) return -JLO_EINVAL;
  int g = Hq / Hkv;
  int64_t kvh = h / g;
  int64_t G = jlo_group_size(L, w_pretrained);
  keyset_t ks;
  const uint16_t* kbase = k + ((int64_t)b * L * Hkv + kvh) * d;
  const uint16_t* vbase = v + ((int64_t)b * L * Hkv + kvh) * d;
  if (keyset_build(&ks, kbase, vbase, qpos + 1, d, (int64_t)Hkv * d, G, theta, 1, NULL) != JLO_OK) {
    keyset_free(&ks);
    return -JLO_ENOMEM;
  }
  double scale = 1.0 / sqrt((double)d);
  double* xq = (double*)malloc(sizeof(double) * (size_t)d);
  double* qb = (double*)malloc(sizeof(double) * (size_t)d);
  double* qr = (double*)malloc(sizeof(double) * (size_t)d);
  double* s = (double*)malloc(sizeof(double) * (size_t)(qpos + 1));
  const double** vv = (const double**)malloc(sizeof(double*) * (size_t)(qpos + 1));
  const uint16_t* qsrc = q + ((b * L + qpos) * Hq + h) * d;
  for (int c = 0; c < d; ++c) xq[c] = bf16_to_double(qsrc[c]);
  jlo_rope_rotate(xq, d, (double)qpos, theta, qb);
  jlo_rope_rotate(xq, d, (double)jlo_remote_position(qpos, G), theta, qr);
  int64_t lo = qpos - w0 < 0 ? 0 : qpos - w0;
  int64_t na = qpos - lo + 1;
  for (int64_t j = 0; j < na; ++j) {
    s[j] = dot(qb, ks.kb + (lo + j) * d, d) * scale;
    vv[j] = ks.v + (lo + j) * d;
  }
  lse3[0] = softmax_call(s, vv, na, d, o3);
  for (int64_t j = 0; j <= qpos; ++j) {
    s[j] = dot(qr, ks.kr + j * d, d) * scale;
    vv[j] = ks.v + j * d;
  }
  lse3[1] = softmax_call(s, vv, qpos + 1, d, o3 + d);
  for (int64_t j = 0; j < na; ++j) {
    s[j] = dot(qr, ks.kr + (lo + j) * d, d) * scale;
    vv[j] = ks.v + (lo + j) * d;
  }
  lse3[2] = softmax_call(s, vv, na, d, o3 + 2 * d);
  free(xq); free(qb); free(qr); free(s); free(vv);
  keyset_free(&ks);
  return JLO_OK;
}

int jlo_max_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}
