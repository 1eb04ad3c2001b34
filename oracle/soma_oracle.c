/*
 * soma_oracle.c -- plain, slow CPU oracle for the SOMA SPSA step.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, loads or
 * calls this file; only the test suite, the smoke check and the benchmark's
 * CPU-baseline leg use it.  It shares no code, header, table or constant
 * generator with the HIP path: both sides implement the same published
 * definitions independently.
 *
 * What it computes (paper, arXiv 2609.37899):
 *   - the central-difference SPSA estimator
 *       g_hat = (1/P) sum_j [(L(theta + eps z_j) - L(theta - eps z_j)) / (2 eps)] z_j
 *     (Section 4, Eq. main-spsa; Appendix E, Eq. localspsa), with every
 *     direction and both signs evaluated on one shared batch (Section 4);
 *   - the separable per-expert loss: expert e is estimated from its own L_e
 *     only (Section 4; Appendix F, Eq. separable-training-objective), or, in
 *     SUMMED mode, from sum_e L_e (Appendix J, independent-vs-summed losses);
 *   - the next-byte cross entropy L_CE(h) = log sum_v exp(w_v . h) - w_y . h
 *     (Appendix E), averaged over all targets, in nats;
 *   - a plain stacked LSTM byte model: embedding -> LSTM_1 -> ... -> LSTM_L ->
 *     linear head (the experts' recurrent body, Section 3 and Appendix C),
 *     bias-free as in Appendix C, gates in the order i, f, g, o;
 *   - the paper's expert body (arch 1: pre-norm residual LSTM and GELU-MLP
 *     blocks with gain-only LayerNorm and the frozen tied E, Appendix C) and
 *     the body of its wider fixed-size controls (arch 2: the same blocks at
 *     width d_t between input and output projections to the head width d_E,
 *     with each expert's own tied E, Appendix C and E), and the decoder-path
 *     delta rule for E (Appendix E, Eq. delta);
 *   - the update theta' = theta - lr * g_hat (plain SGD step on g_hat) and the
 *     paper's Adam-style update with coupled weight decay (Appendix E).
 *
 * Probe laws (cfg.probe), all from counter-based Philox4x32-10 (Salmon,
 * Moraes, Dror, Shaw, SC'11, "Parallel random numbers: as easy as 1, 2, 3"):
 *   0  Gaussian: z ~ N(0,1) per parameter by the Box-Muller transform.  The
 *      logarithm and the sine/cosine it uses are this file's own fp32
 *      routines (series below), a fixed sequence of correctly rounded IEEE
 *      operations, reproducible bit for bit on any conforming machine.
 *   1  sparse Rademacher, the paper's training law (Appendix E): each
 *      coordinate is 0 with probability 1/2 and -1 or +1 with probability
 *      1/4 each; the normalization gains of arch 1 and 2 are always +-1
 *      (Appendix E).
 *   2  dense Rademacher, the law of the paper's variance theory (Section 4,
 *      Eq. main-spsa; Appendix F, Prop. block-variance): -1 or +1 with
 *      probability 1/2 each.
 *   Both Rademacher laws read a 2-bit field per coordinate (64 coordinates
 *   per Philox block): the high bit says whether a sparse coordinate is
 *   active, the low bit is the sign (1 = -1).  The dense law uses the sign
 *   bit alone, so the two laws agree wherever the sparse one is nonzero.
 *
 * Precision: perturbed weights are formed in fp32 with one rounding
 * (fmaf(+-eps, z, theta)); the forward pass, the losses, the coefficients and
 * the update sum are carried in fp64; theta' is rounded once to fp32.
 *
 * Build: cc -O2 -std=c11 -fopenmp -ffp-contract=off -fno-fast-math -shared
 *        -fPIC -o liboracle.so soma_oracle.c -lm
 * (contraction must stay off: the RNG is specified operation by operation).
 */
#define _POSIX_C_SOURCE 200809L
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* ------------------------------------------------------------------------ */
/* Model configuration (the oracle's own definition).                        */
/* ------------------------------------------------------------------------ */
typedef struct {
  int32_t n_experts; /* N */
  int32_t n_layers;  /* L */
  int32_t embed;     /* E */
  int32_t hidden;    /* H */
  int32_t batch;     /* B sequences per expert */
  int32_t seq_len;   /* T bytes per sequence -> T-1 targets */
  int32_t n_pairs;   /* P antithetic pairs (directions) per expert */
  int32_t loss_mode; /* 0: independent per-expert losses, 1: summed loss */
  int32_t probe;     /* probe law: 0 Gaussian, 1 sparse Rademacher, 2 dense Rademacher */
  int32_t accum;     /* A accumulation batches per update (0 or 1: one batch) */
  int32_t arch;      /* 0: stacked LSTM + linear head; 1: the paper's expert body; 2: the body of
                        the wide controls (both below) */
  const float *tied_head; /* arch 1, 2: the tied embedding/decoder E [V][head width] of expert 0 */
  int64_t head_stride;    /* floats from one expert's E to the next (0: one shared E) */
  uint32_t perturb_mask;  /* perturbed parameter groups: bit 0 embedding, bit 1 LSTM layers (the
                             whole body for arch 1), bit 2 head; 0 means all of them */
} oracle_cfg;

/* Directions per update: P per batch, A batches. */
static int total_dirs(const oracle_cfg *c) { return c->n_pairs * (c->accum > 1 ? c->accum : 1); }

#define VOCAB 256

/* Canonical flat layout of one expert's parameter vector:
 *   Emb[V][E]; for l = 1..L: W_l[4H][in_l + H] (rows: gate blocks i,f,g,o;
 *   columns: [input | recurrent]), in_1 = E, in_l = H; Whead[V][H].          */
static int64_t in_dim(const oracle_cfg *c, int l) { return l == 0 ? c->embed : c->hidden; }

static int64_t off_layer(const oracle_cfg *c, int l) {
  int64_t off = (int64_t)VOCAB * c->embed;
  for (int i = 0; i < l; ++i) off += 4LL * c->hidden * (in_dim(c, i) + c->hidden);
  return off;
}

/* The paper's expert body (arch 1; Section 3 and Appendix C, Fig. arch):
 * width d = embed = hidden; D = n_layers pre-norm residual blocks, each an
 * LSTM sublayer and a GELU MLP (hidden 4d), both bias-free, with gain-only
 * LayerNorm; a final gain-only LayerNorm; the frozen tied matrix E embeds the
 * input byte and decodes logits = LN(x) E^T.  E is not part of theta.
 * Body layout (canonical k), per block l: g1[d]; W[4d][2d] (gates i,f,g,o;
 * columns [input | recurrent]); g2[d]; W1[4d][d]; W2[d][4d]; then g_f[d]:
 * d_body = D (16 d^2 + 2 d) + d (the paper's 16 D d_t^2 + (2D + 1) d_t).
 * LayerNorm(x; g) = g (x - mean) / sqrt(var + 1e-5) (biased variance over
 * the d features); GELU(u) = u Phi(u) = u (1 + erf(u / sqrt 2)) / 2. */
#define LN_EPS 1e-5

static int64_t body_block(int64_t d) { return 16 * d * d + 2 * d; }

/* The body of the wider fixed-size controls (arch 2; Appendix C, counting
 * rules and Table fixed-parameter-counts): the same D blocks at width
 * d_t = hidden, between input and output projections to the head width
 * d_E = embed, so the count is 16 D d_t^2 + (2D + 1) d_t + 2 d_E d_t.  The
 * head E [V][d_E] is tied between input and output within an expert, local
 * to it and never perturbed (Appendix E): x_0 = P_in E[byte]; the blocks as
 * in arch 1; f = LayerNorm(x; g_f); the decoder input is u = P_out f and the
 * logits are E u.  Where the projections sit is fixed only by the count; the
 * reading here puts them at the two ends of the body.
 * Layout (canonical k; every matrix row a multiple of 4 long, so that a probe
 * quad never straddles two rows):
 *   P_in [d_t][d_E]             x_0[c] = sum_q P_in[c][q] E[byte][q]
 *   per block l:
 *     A_l [d_t][4 d_t]          LSTM input weights, a[j] = sum_c n[c] A_l[c][j]
 *     R_l [d_t][4 d_t]          LSTM recurrent weights, a[j] += sum_c h[c] R_l[c][j]
 *                               (j = gate g d_t + unit, gates i, f, g, o)
 *     U_l [d_t][4 d_t]          MLP up, m[j] = GELU(sum_c n[c] U_l[c][j])
 *     V_l [d_t][4 d_t]          MLP down, x[c] += sum_j V_l[c][j] m[j]
 *   P_out [d_t][d_E]            u[q] = sum_c f[c] P_out[c][q]
 *   gains: g1_l, g2_l for l = 1..D, then g_f (each d_t long)            */
static int64_t wide_off_block(const oracle_cfg *c, int l) {
  const int64_t d = c->hidden;
  return d * c->embed + (int64_t)l * 16 * d * d;
}
static int64_t wide_off_gain(const oracle_cfg *c) {
  return wide_off_block(c, c->n_layers) + (int64_t)c->hidden * c->embed;
}

int64_t oracle_param_count(const oracle_cfg *c) {
  if (c->arch == 1) return c->n_layers * body_block(c->hidden) + c->hidden;
  if (c->arch == 2) return wide_off_gain(c) + (2LL * c->n_layers + 1) * c->hidden;
  return off_layer(c, c->n_layers) + (int64_t)VOCAB * c->hidden;
}

/* Width of the tied head E: d = d_t for arch 1, d_E for arch 2. */
static int head_width(const oracle_cfg *c) { return c->arch == 2 ? c->embed : c->hidden; }

/* Whether coordinate k of the body is a LayerNorm gain. */
static int body_is_gain(const oracle_cfg *c, int64_t k) {
  if (c->arch == 2) return k >= wide_off_gain(c);
  const int64_t d = c->hidden, blk = body_block(d);
  if (k >= c->n_layers * blk) return 1;               /* g_f */
  const int64_t r = k % blk;
  return r < d || (r >= d + 8 * d * d && r < 2 * d + 8 * d * d);
}

/* Whether coordinate k is perturbed and updated (cfg.perturb_mask).  The
 * paper keeps parts of the model out of the search: its decoder/embedding E
 * is never perturbed and only the body is (Section 4; Appendix E).  For the
 * stacked LSTM the groups are the embedding (bit 0), the LSTM layers (bit 1)
 * and the head (bit 2); the body of arch 1 or 2 is one group (bit 1).  A
 * masked coordinate keeps its value in every perturbed forward and in the
 * update. */
static int coord_perturbed(const oracle_cfg *c, int64_t k) {
  const uint32_t m = c->perturb_mask ? c->perturb_mask : 7u;
  if (c->arch != 0) return (int)((m >> 1) & 1u);
  const int grp = k < (int64_t)VOCAB * c->embed ? 0 : (k < off_layer(c, c->n_layers) ? 1 : 2);
  return (int)((m >> grp) & 1u);
}

/* The probe law of coordinate k: under the paper's sparse law its
 * normalization gains are dense +-1 (Appendix E); otherwise the configured law. */
static int law_of(const oracle_cfg *c, int64_t k) {
  return (c->arch != 0 && c->probe == 1 && body_is_gain(c, k)) ? 2 : c->probe;
}

/* ------------------------------------------------------------------------ */
/* Philox4x32-10 (SC'11).  One round maps (c0,c1,c2,c3) with key (k0,k1) to  */
/*   (hi(M1*c2) ^ c1 ^ k0, lo(M1*c2), hi(M0*c0) ^ c3 ^ k1, lo(M0*c0));        */
/* the key is advanced by the Weyl constants between rounds.                 */
/* ------------------------------------------------------------------------ */
#define PHILOX_M0 0xD2511F53u
#define PHILOX_M1 0xCD9E8D57u
#define PHILOX_W0 0x9E3779B9u
#define PHILOX_W1 0xBB67AE85u

void oracle_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]) {
  uint32_t x0 = ctr[0], x1 = ctr[1], x2 = ctr[2], x3 = ctr[3];
  uint32_t k0 = key[0], k1 = key[1];
  for (int round = 0; round < 10; ++round) {
    if (round > 0) {
      k0 += PHILOX_W0;
      k1 += PHILOX_W1;
    }
    uint64_t p0 = (uint64_t)PHILOX_M0 * (uint64_t)x0;
    uint64_t p1 = (uint64_t)PHILOX_M1 * (uint64_t)x2;
    uint32_t y0 = (uint32_t)(p1 >> 32) ^ x1 ^ k0;
    uint32_t y1 = (uint32_t)p1;
    uint32_t y2 = (uint32_t)(p0 >> 32) ^ x3 ^ k1;
    uint32_t y3 = (uint32_t)p0;
    x0 = y0; x1 = y1; x2 = y2; x3 = y3;
  }
  out[0] = x0; out[1] = x1; out[2] = x2; out[3] = x3;
}

/* ------------------------------------------------------------------------ */
/* Own fp32 elementary functions for Box-Muller.                              */
/*                                                                            */
/* Series coefficients are the fp32 values nearest to the exact reals        */
/*   S_n = (-1)^((n-1)/2) (pi/2)^n / n!  (n odd)   -- sin(pi/2 r)            */
/*   C_n = (-1)^(n/2)     (pi/2)^n / n!  (n even)  -- cos(pi/2 r)            */
/* computed here from that definition in double and rounded once.            */
/* ------------------------------------------------------------------------ */
static float g_sin_c[6];  /* S1, S3, S5, S7, S9, S11 */
static float g_cos_c[7];  /* C0, C2, ..., C12 */

__attribute__((constructor)) static void oracle_init_constants(void) {
  const double half_pi = 1.57079632679489661923132169163975144;
  for (int i = 0; i < 6; ++i) {
    int n = 2 * i + 1;
    double v = 1.0;
    for (int m = 1; m <= n; ++m) v = v * half_pi / (double)m;
    g_sin_c[i] = (float)((i & 1) ? -v : v);
  }
  for (int i = 0; i < 7; ++i) {
    int n = 2 * i;
    double v = 1.0;
    for (int m = 1; m <= n; ++m) v = v * half_pi / (double)m;
    g_cos_c[i] = (float)((i & 1) ? -v : v);
  }
}

/* Expose the coefficient table for the pin test (S1..S11 then C0..C12). */
void oracle_series_constants(float out[13]) {
  for (int i = 0; i < 6; ++i) out[i] = g_sin_c[i];
  for (int i = 0; i < 7; ++i) out[6 + i] = g_cos_c[i];
}

/* ln(m * 2^-24) for integer m in [1, 2^24], in fp32.
 * Method: write m 2^-24 = 2^n f with f in (sqrt(1/2), sqrt(2)]; then
 * ln f = 2 atanh(s), s = (f-1)/(f+1), |s| <= 0.1716, and
 * 2 atanh(s) = 2s (1 + s^2/3 + s^4/5 + s^6/7 + s^8/9 + s^10/11 + ...).
 * ln 2 is split Cody-Waite style into a 16-bit head (exact products n*hi)
 * and a tail. */
float oracle_ln_u24(uint32_t m) {
  int e = 31 - __builtin_clz(m);           /* floor(log2 m), 0..24 */
  float f = ldexpf((float)m, -e);          /* exact, in [1, 2) */
  if (f > 0x1.6a09e6p+0f) {                /* fp32 nearest to sqrt(2) */
    f = f * 0.5f;
    e = e + 1;
  }
  const float n = (float)(e - 24);
  const float ln2_hi = 0.693145751953125f;                               /* 0x3F317200 */
  const float ln2_lo = (float)(0.69314718055994530942 - 0.693145751953125);
  float s = (f - 1.0f) / (f + 1.0f);
  float s2 = s * s;
  float q = fmaf(s2, 1.0f / 11.0f, 1.0f / 9.0f);
  q = fmaf(s2, q, 1.0f / 7.0f);
  q = fmaf(s2, q, 1.0f / 5.0f);
  q = fmaf(s2, q, 1.0f / 3.0f);
  q = q * s2;
  float two_s = s + s;
  float lnf = fmaf(two_s, q, two_s);
  return fmaf(n, ln2_hi, fmaf(n, ln2_lo, lnf));
}

/* cos and sin of 2 pi i 2^-24 for integer i in [0, 2^24).
 * Quarter-turn reduction is exact: 4 i 2^-24 = qd + r with qd the nearest
 * integer (ties up) and r in [-1/2, 1/2); angle = pi/2 (qd + r).            */
void oracle_sincos_2pi_u24(uint32_t i, float *c_out, float *s_out) {
  uint32_t qd = (i + (1u << 21)) >> 22;               /* 0..4 */
  int32_t rem = (int32_t)i - (int32_t)(qd << 22);     /* [-2^21, 2^21) */
  float r = (float)rem * 0x1p-22f;                    /* exact */
  float r2 = r * r;
  float sp = fmaf(r2, g_sin_c[5], g_sin_c[4]);
  sp = fmaf(r2, sp, g_sin_c[3]);
  sp = fmaf(r2, sp, g_sin_c[2]);
  sp = fmaf(r2, sp, g_sin_c[1]);
  sp = fmaf(r2, sp, g_sin_c[0]);
  float sn = sp * r;                                  /* sin(pi/2 r) */
  float cp = fmaf(r2, g_cos_c[6], g_cos_c[5]);
  cp = fmaf(r2, cp, g_cos_c[4]);
  cp = fmaf(r2, cp, g_cos_c[3]);
  cp = fmaf(r2, cp, g_cos_c[2]);
  cp = fmaf(r2, cp, g_cos_c[1]);
  float cs = fmaf(r2, cp, g_cos_c[0]);                /* cos(pi/2 r) */
  float c, s;
  switch (qd & 3u) {
    case 0: c = cs;  s = sn;  break;
    case 1: c = -sn; s = cs;  break;
    case 2: c = -cs; s = -sn; break;
    default: c = sn; s = -cs; break;
  }
  *c_out = c;
  *s_out = s;
}

/* Box-Muller on one pair of Philox words (wa, wb):
 *   u1 = ((wa >> 8) + 1) 2^-24 in (0, 1],  u2 = (wb >> 8) 2^-24 in [0, 1),
 *   r = sqrt(-2 ln u1),  za = r cos(2 pi u2),  zb = r sin(2 pi u2).         */
void oracle_box_muller(uint32_t wa, uint32_t wb, float *za, float *zb) {
  float lnu = oracle_ln_u24((wa >> 8) + 1u);
  float r = sqrtf(-2.0f * lnu);
  float c, s;
  oracle_sincos_2pi_u24(wb >> 8, &c, &s);
  *za = r * c;
  *zb = r * s;
}

/* Array forms of the two routines above, for the exhaustive pin tests. */
void oracle_ln_u24_array(const uint32_t *m, int64_t n, float *out) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) out[i] = oracle_ln_u24(m[i]);
}

void oracle_sincos_2pi_u24_array(const uint32_t *idx, int64_t n, float *c, float *s) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) oracle_sincos_2pi_u24(idx[i], &c[i], &s[i]);
}

void oracle_box_muller_array(const uint32_t *wa, const uint32_t *wb, int64_t n, float *za,
                             float *zb) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) oracle_box_muller(wa[i], wb[i], &za[i], &zb[i]);
}

/* The four Gaussians z[4q .. 4q+3] of direction `pair` at SPSA step `step`
 * for an expert whose stream seed is `seed`.
 *   key     = (lo32(seed), hi32(seed) ^ hi32(step))
 *   counter = (lo32(q), pair, lo32(step), hi32(q))
 *   (w0, w1) -> z[4q], z[4q+1];  (w2, w3) -> z[4q+2], z[4q+3].            */
static void gaussian_quad(uint64_t seed, uint64_t step, uint32_t pair, uint64_t q, float z[4]) {
  uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32) ^ (uint32_t)(step >> 32)};
  uint32_t ctr[4] = {(uint32_t)q, pair, (uint32_t)step, (uint32_t)(q >> 32)};
  uint32_t w[4];
  oracle_philox4x32_10(ctr, key, w);
  oracle_box_muller(w[0], w[1], &z[0], &z[1]);
  oracle_box_muller(w[2], w[3], &z[2], &z[3]);
}

void oracle_gaussian(uint64_t seed, uint64_t step, uint32_t pair, uint64_t k0, uint64_t count,
                     float *out) {
  for (uint64_t i = 0; i < count; ++i) {
    uint64_t k = k0 + i;
    float z[4];
    gaussian_quad(seed, step, pair, k >> 2, z);
    out[i] = z[k & 3];
  }
}

/* Rademacher probe value of coordinate k (laws 1 and 2).
 *   key     = (lo32(seed), hi32(seed) ^ hi32(step))          (as above)
 *   counter = (lo32(b), pair, lo32(step), hi32(b)),  b = k >> 6
 *   field   = bits 2 (k & 15) .. +1 of word (k >> 4) & 3 of the block's output. */
static float rademacher_value(int law, uint64_t seed, uint64_t step, uint32_t pair, uint64_t k) {
  const uint64_t b = k >> 6;
  uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32) ^ (uint32_t)(step >> 32)};
  uint32_t ctr[4] = {(uint32_t)b, pair, (uint32_t)step, (uint32_t)(b >> 32)};
  uint32_t w[4];
  oracle_philox4x32_10(ctr, key, w);
  const uint32_t field = (w[(k >> 4) & 3] >> (2 * (k & 15))) & 3u;
  const float sgn = (field & 1u) ? -1.0f : 1.0f;
  if (law == 2) return sgn;
  return (field >> 1) ? sgn : 0.0f;
}

/* z_pair[4q .. 4q+3] under probe law `law`. */
static void probe_quad(int law, uint64_t seed, uint64_t step, uint32_t pair, uint64_t q, float z[4]) {
  if (law == 0) {
    gaussian_quad(seed, step, pair, q, z);
    return;
  }
  for (int i = 0; i < 4; ++i) z[i] = rademacher_value(law, seed, step, pair, 4 * q + (uint64_t)i);
}

/* count probe values z_pair[k0 .. k0+count) under law `law` (0, 1 or 2). */
int oracle_probe(int law, uint64_t seed, uint64_t step, uint32_t pair, uint64_t k0, uint64_t count,
                 float *out) {
  if (law < 0 || law > 2) return -1;
  for (uint64_t i = 0; i < count; ++i) {
    uint64_t k = k0 + i;
    float z[4];
    probe_quad(law, seed, step, pair, k >> 2, z);
    out[i] = z[k & 3];
  }
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Forward pass and loss, fp64.                                               */
/* ------------------------------------------------------------------------ */
static double sigmoid(double x) { return 1.0 / (1.0 + exp(-x)); }

/* Sum of next-byte cross entropies of one sequence (T-1 targets). */
static double sequence_ce_sum(const oracle_cfg *c, const double *w, const uint8_t *seq,
                              double *scratch) {
  const int L = c->n_layers, E = c->embed, H = c->hidden, T = c->seq_len;
  double *h = scratch;                 /* [L][H] */
  double *cs = h + (size_t)L * H;      /* [L][H] */
  double *x = cs + (size_t)L * H;      /* [max(E,H)] */
  double *a = x + (E > H ? E : H);     /* [4H] */
  double *logits = a + 4 * (size_t)H;  /* [V] */
  memset(h, 0, sizeof(double) * 2 * (size_t)L * H);
  const double *emb = w;
  const double *head = w + off_layer(c, L);
  double total = 0.0;
  for (int t = 0; t + 1 < T; ++t) {
    const double *erow = emb + (size_t)seq[t] * E;
    for (int k = 0; k < E; ++k) x[k] = erow[k];
    int xin = E;
    for (int l = 0; l < L; ++l) {
      const double *W = w + off_layer(c, l);
      const int cols = xin + H;
      double *hl = h + (size_t)l * H, *cl = cs + (size_t)l * H;
      for (int r = 0; r < 4 * H; ++r) {
        const double *wr = W + (size_t)r * cols;
        double acc = 0.0;
        for (int k = 0; k < xin; ++k) acc += wr[k] * x[k];
        for (int k = 0; k < H; ++k) acc += wr[xin + k] * hl[k];
        a[r] = acc;
      }
      for (int u = 0; u < H; ++u) {
        double ig = sigmoid(a[u]);
        double fg = sigmoid(a[H + u]);
        double gg = tanh(a[2 * H + u]);
        double og = sigmoid(a[3 * H + u]);
        cl[u] = fg * cl[u] + ig * gg;
        hl[u] = og * tanh(cl[u]);
      }
      for (int u = 0; u < H; ++u) x[u] = hl[u];
      xin = H;
    }
    double mx = -INFINITY;
    for (int v = 0; v < VOCAB; ++v) {
      const double *wr = head + (size_t)v * H;
      double acc = 0.0;
      for (int k = 0; k < H; ++k) acc += wr[k] * x[k];
      logits[v] = acc;
      if (acc > mx) mx = acc;
    }
    double se = 0.0;
    for (int v = 0; v < VOCAB; ++v) se += exp(logits[v] - mx);
    total += log(se) + mx - logits[seq[t + 1]];
  }
  return total;
}

static void layer_norm(const double *x, const double *g, int d, double *out) {
  double mu = 0.0, var = 0.0;
  for (int k = 0; k < d; ++k) mu += x[k];
  mu /= d;
  for (int k = 0; k < d; ++k) var += (x[k] - mu) * (x[k] - mu);
  var /= d;
  const double inv = 1.0 / sqrt(var + LN_EPS);
  for (int k = 0; k < d; ++k) out[k] = g[k] * (x[k] - mu) * inv;
}

static double gelu(double u) { return 0.5 * u * (1.0 + erf(u / sqrt(2.0))); }

/* Sum of next-byte cross entropies of one sequence under the paper's body
 * (arch 1), E the frozen tied matrix [V][d] (fp64).  When dE != NULL the
 * decoder-path derivative (p - onehot(y)) f^T of every target, f the decoder
 * input, is added to dE [V][d] (Appendix E, Eq. delta, before the mean). */
static double sequence_ce_sum_body(const oracle_cfg *c, const double *w, const double *E, const uint8_t *seq,
                                   double *scratch, double *dE) {
  const int D = c->n_layers, d = c->hidden, T = c->seq_len;
  const int64_t blk = body_block(d);
  double *h = scratch;                  /* [D][d] */
  double *cs = h + (size_t)D * d;       /* [D][d] */
  double *x = cs + (size_t)D * d;       /* [d] */
  double *n = x + d;                    /* [d] */
  double *a = n + d;                    /* [4d] */
  double *u = a + 4 * (size_t)d;        /* [4d] */
  double *logits = u + 4 * (size_t)d;   /* [V] */
  memset(h, 0, sizeof(double) * 2 * (size_t)D * d);
  const double *gf = w + D * blk;
  double total = 0.0;
  for (int t = 0; t + 1 < T; ++t) {
    for (int k = 0; k < d; ++k) x[k] = E[(size_t)seq[t] * d + k];
    for (int l = 0; l < D; ++l) {
      const double *g1 = w + l * blk, *W = g1 + d, *g2 = W + 8 * (size_t)d * d;
      const double *W1 = g2 + d, *W2 = W1 + 4 * (size_t)d * d;
      double *hl = h + (size_t)l * d, *cl = cs + (size_t)l * d;
      layer_norm(x, g1, d, n);                                   /* LSTM sublayer */
      for (int r = 0; r < 4 * d; ++r) {
        const double *wr = W + (size_t)r * 2 * d;
        double acc = 0.0;
        for (int k = 0; k < d; ++k) acc += wr[k] * n[k];
        for (int k = 0; k < d; ++k) acc += wr[d + k] * hl[k];
        a[r] = acc;
      }
      for (int q = 0; q < d; ++q) {
        const double ig = sigmoid(a[q]), fg = sigmoid(a[d + q]), gg = tanh(a[2 * d + q]),
                     og = sigmoid(a[3 * d + q]);
        cl[q] = fg * cl[q] + ig * gg;
        hl[q] = og * tanh(cl[q]);
      }
      for (int k = 0; k < d; ++k) x[k] += hl[k];                 /* residual */
      layer_norm(x, g2, d, n);                                   /* MLP sublayer */
      for (int r = 0; r < 4 * d; ++r) {
        const double *wr = W1 + (size_t)r * d;
        double acc = 0.0;
        for (int k = 0; k < d; ++k) acc += wr[k] * n[k];
        u[r] = gelu(acc);
      }
      for (int r = 0; r < d; ++r) {
        const double *wr = W2 + (size_t)r * 4 * d;
        double acc = 0.0;
        for (int k = 0; k < 4 * d; ++k) acc += wr[k] * u[k];
        x[r] += acc;                                             /* residual */
      }
    }
    layer_norm(x, gf, d, n);                                     /* decoder input f */
    double mx = -INFINITY;
    for (int v = 0; v < VOCAB; ++v) {
      double acc = 0.0;
      for (int k = 0; k < d; ++k) acc += E[(size_t)v * d + k] * n[k];
      logits[v] = acc;
      if (acc > mx) mx = acc;
    }
    double se = 0.0;
    for (int v = 0; v < VOCAB; ++v) se += exp(logits[v] - mx);
    const int y = seq[t + 1];
    total += log(se) + mx - logits[y];
    if (dE)
      for (int v = 0; v < VOCAB; ++v) {
        const double pv = exp(logits[v] - mx) / se - (v == y ? 1.0 : 0.0);
        for (int k = 0; k < d; ++k) dE[(size_t)v * d + k] += pv * n[k];
      }
  }
  return total;
}

/* Sum of next-byte cross entropies of one sequence under the wide controls'
 * body (arch 2), E the expert's tied matrix [V][d_E] (fp64).  When dE != NULL
 * the decoder-path derivative (p - onehot(y)) u^T of every target, u the
 * decoder input, is added to dE [V][d_E] (Appendix E, Eq. delta). */
static double sequence_ce_sum_wide(const oracle_cfg *c, const double *w, const double *E, const uint8_t *seq,
                                   double *scratch, double *dE) {
  const int D = c->n_layers, d = c->hidden, dE_ = c->embed, T = c->seq_len;
  const int64_t d4 = 4 * (int64_t)d;
  double *h = scratch;                  /* [D][d] */
  double *cs = h + (size_t)D * d;       /* [D][d] */
  double *x = cs + (size_t)D * d;       /* [d] */
  double *n = x + d;                    /* [d] */
  double *a = n + d;                    /* [4d] */
  double *m = a + d4;                   /* [4d] */
  double *u = m + d4;                   /* [d_E] */
  double *logits = u + dE_;             /* [V] */
  memset(h, 0, sizeof(double) * 2 * (size_t)D * d);
  const double *Pin = w, *Pout = w + wide_off_block(c, D), *gains = w + wide_off_gain(c);
  const double *gf = gains + 2 * (size_t)D * d;
  double total = 0.0;
  for (int t = 0; t + 1 < T; ++t) {
    const double *ey = E + (size_t)seq[t] * dE_;
    for (int k = 0; k < d; ++k) {                               /* input projection */
      double acc = 0.0;
      for (int q = 0; q < dE_; ++q) acc += Pin[(size_t)k * dE_ + q] * ey[q];
      x[k] = acc;
    }
    for (int l = 0; l < D; ++l) {
      const double *A = w + wide_off_block(c, l), *R = A + d4 * d, *U = R + d4 * d, *Vd = U + d4 * d;
      const double *g1 = gains + 2 * (size_t)l * d, *g2 = g1 + d;
      double *hl = h + (size_t)l * d, *cl = cs + (size_t)l * d;
      layer_norm(x, g1, d, n);                                   /* LSTM sublayer */
      for (int64_t j = 0; j < d4; ++j) {
        double acc = 0.0;
        for (int k = 0; k < d; ++k) acc += n[k] * A[(size_t)k * d4 + j];
        for (int k = 0; k < d; ++k) acc += hl[k] * R[(size_t)k * d4 + j];
        a[j] = acc;
      }
      for (int q = 0; q < d; ++q) {
        const double ig = sigmoid(a[q]), fg = sigmoid(a[d + q]), gg = tanh(a[2 * d + q]),
                     og = sigmoid(a[3 * d + q]);
        cl[q] = fg * cl[q] + ig * gg;
        hl[q] = og * tanh(cl[q]);
      }
      for (int k = 0; k < d; ++k) x[k] += hl[k];                 /* residual */
      layer_norm(x, g2, d, n);                                   /* MLP sublayer */
      for (int64_t j = 0; j < d4; ++j) {
        double acc = 0.0;
        for (int k = 0; k < d; ++k) acc += n[k] * U[(size_t)k * d4 + j];
        m[j] = gelu(acc);
      }
      for (int k = 0; k < d; ++k) {
        double acc = 0.0;
        for (int64_t j = 0; j < d4; ++j) acc += Vd[(size_t)k * d4 + j] * m[j];
        x[k] += acc;                                             /* residual */
      }
    }
    layer_norm(x, gf, d, n);                                     /* f */
    for (int q = 0; q < dE_; ++q) {                              /* output projection: u */
      double acc = 0.0;
      for (int k = 0; k < d; ++k) acc += n[k] * Pout[(size_t)k * dE_ + q];
      u[q] = acc;
    }
    double mx = -INFINITY;
    for (int v = 0; v < VOCAB; ++v) {
      double acc = 0.0;
      for (int q = 0; q < dE_; ++q) acc += E[(size_t)v * dE_ + q] * u[q];
      logits[v] = acc;
      if (acc > mx) mx = acc;
    }
    double se = 0.0;
    for (int v = 0; v < VOCAB; ++v) se += exp(logits[v] - mx);
    const int y = seq[t + 1];
    total += log(se) + mx - logits[y];
    if (dE)
      for (int v = 0; v < VOCAB; ++v) {
        const double pv = exp(logits[v] - mx) / se - (v == y ? 1.0 : 0.0);
        for (int q = 0; q < dE_; ++q) dE[(size_t)v * dE_ + q] += pv * u[q];
      }
  }
  return total;
}

static double sequence_ce_sum_head(const oracle_cfg *c, const double *w, const double *E, const uint8_t *seq,
                                   double *scratch, double *dE) {
  return c->arch == 2 ? sequence_ce_sum_wide(c, w, E, seq, scratch, dE)
                      : sequence_ce_sum_body(c, w, E, seq, scratch, dE);
}

static size_t scratch_doubles(const oracle_cfg *c);

static double *head_f64(const oracle_cfg *c) {
  const size_t nE = (size_t)VOCAB * head_width(c);
  double *E = (double *)malloc(sizeof(double) * nE);
  for (size_t i = 0; i < nE; ++i) E[i] = (double)c->tied_head[i];
  return E;
}

/* The decoder-path derivative of the unperturbed mean cross entropy with
 * respect to the tied matrix (Appendix E, Eq. delta), one expert (arch 1 or 2):
 *   dE = (1 / (B (T-1))) sum_{b,t} (p_{b,t} - onehot(y_{b,t+1})) f_{b,t}^T,
 * holding the decoder inputs f fixed (f = LayerNorm(x; g_f) for arch 1, the
 * output projection u for arch 2).  grad [V][head width] fp64 out.  Returns
 * the mean cross entropy, or NaN for a configuration without a tied head. */
double oracle_head_delta(const oracle_cfg *c, const float *theta, const uint8_t *bytes, double *grad) {
  if ((c->arch != 1 && c->arch != 2) || !c->tied_head) return NAN;
  const int B = c->batch, T = c->seq_len, d = head_width(c);
  const int64_t nd = oracle_param_count(c);
  double *w = (double *)malloc(sizeof(double) * (size_t)nd);
  for (int64_t k = 0; k < nd; ++k) w[k] = (double)theta[k];
  double *E = head_f64(c);
  double *scratch = (double *)malloc(sizeof(double) * scratch_doubles(c));
  memset(grad, 0, sizeof(double) * (size_t)VOCAB * d);
  double total = 0.0;
  for (int b = 0; b < B; ++b) total += sequence_ce_sum_head(c, w, E, bytes + (size_t)b * T, scratch, grad);
  const double inv = 1.0 / ((double)B * (double)(T - 1));
  for (size_t i = 0; i < (size_t)VOCAB * d; ++i) grad[i] *= inv;
  free(scratch);
  free(E);
  free(w);
  return total * inv;
}

static size_t scratch_doubles(const oracle_cfg *c) {
  const size_t L = c->n_layers, E = c->embed, H = c->hidden;
  if (c->arch == 1) return 2 * L * H + 10 * H + VOCAB;
  if (c->arch == 2) return 2 * L * H + 10 * H + E + VOCAB;
  return 2 * L * H + (E > H ? E : H) + 4 * H + VOCAB;
}

/* Mean cross entropy (nats per target byte) of one model with fp64 weights
 * over its B sequences of T bytes.  Sequences are independent forwards and
 * may run in parallel; their sums are added in sequence order. */
double oracle_forward_loss_f64(const oracle_cfg *c, const double *w, const uint8_t *bytes) {
  const int B = c->batch, T = c->seq_len;
  double *seq_sum = (double *)malloc(sizeof(double) * (size_t)B);
  const size_t ns = scratch_doubles(c);
  double *E = c->arch != 0 ? head_f64(c) : NULL;
#pragma omp parallel
  {
    double *scratch = (double *)malloc(sizeof(double) * ns);
#pragma omp for schedule(dynamic, 1)
    for (int b = 0; b < B; ++b)
      seq_sum[b] = c->arch != 0 ? sequence_ce_sum_head(c, w, E, bytes + (size_t)b * T, scratch, NULL)
                                : sequence_ce_sum(c, w, bytes + (size_t)b * T, scratch);
    free(scratch);
  }
  free(E);
  double total = 0.0;
  for (int b = 0; b < B; ++b) total += seq_sum[b];
  free(seq_sum);
  return total / ((double)B * (double)(T - 1));
}

double oracle_forward_loss(const oracle_cfg *c, const float *w32, const uint8_t *bytes) {
  const int64_t d = oracle_param_count(c);
  double *w = (double *)malloc(sizeof(double) * (size_t)d);
  for (int64_t k = 0; k < d; ++k) w[k] = (double)w32[k];
  double loss = oracle_forward_loss_f64(c, w, bytes);
  free(w);
  return loss;
}

/* w = fl32(theta + s*eps*z_pair) with one rounding, s*eps passed as sign_eps. */
void oracle_perturb(const oracle_cfg *c, const float *theta, uint64_t seed, uint64_t step,
                    uint32_t pair, float sign_eps, float *w_out) {
  const int64_t d = oracle_param_count(c);
  for (int64_t q = 0; 4 * q < d; ++q) {
    float z[4];
    probe_quad(law_of(c, 4 * q), seed, step, pair, (uint64_t)q, z);
    for (int i = 0; i < 4 && 4 * q + i < d; ++i) {
      int64_t k = 4 * q + i;
      w_out[k] = coord_perturbed(c, k) ? fmaf(sign_eps, z[i], theta[k]) : theta[k];
    }
  }
}

/* L(theta + sign*eps*z_pair) for one expert. */
double oracle_perturbed_loss(const oracle_cfg *c, const float *theta, uint64_t seed, uint64_t step,
                             uint32_t pair, int sign, float eps, const uint8_t *bytes) {
  const int64_t d = oracle_param_count(c);
  float *w = (float *)malloc(sizeof(float) * (size_t)d);
  oracle_perturb(c, theta, seed, step, pair, sign >= 0 ? eps : -eps, w);
  double loss = oracle_forward_loss(c, w, bytes);
  free(w);
  return loss;
}

/* ------------------------------------------------------------------------ */
/* SPSA step.                                                                 */
/* ------------------------------------------------------------------------ */

/* Given per-direction coefficients coef[j] = (L+ - L-)/(2 eps P), return
 *   theta'[k] = fl32(theta[k] - lr * sum_j coef[j] z_j[k])   (sum in j order),
 * for the listed coordinates ks[0..nk) (or all when ks == NULL), and the
 * estimate g_hat[k] = sum_j coef[j] z_j[k] when ghat != NULL. */
void oracle_apply_update(const oracle_cfg *c, const float *theta, uint64_t seed, uint64_t step,
                         float lr, const double *coef, const int64_t *ks, int64_t nk,
                         float *theta_out, double *ghat) {
  const int P = total_dirs(c);
  const int64_t n = ks ? nk : oracle_param_count(c);
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) {
    const int64_t k = ks ? ks[i] : i;
    if (!coord_perturbed(c, k)) {          /* masked: no estimate, no update */
      theta_out[i] = theta[k];
      if (ghat) ghat[i] = 0.0;
      continue;
    }
    double g = 0.0;
    for (int j = 0; j < P; ++j) {
      float z[4];
      probe_quad(law_of(c, k & ~(int64_t)3), seed, step, (uint32_t)j, (uint64_t)k >> 2, z);
      g += coef[j] * (double)z[k & 3];
    }
    theta_out[i] = (float)((double)theta[k] - (double)lr * g);
    if (ghat) ghat[i] = g;
  }
}

/* The paper's update (Appendix E, Eq. localspsa, with coupled weight decay):
 *   g  = g_hat + lambda theta                    (decay added before the moments)
 *   m' = beta1 m + (1 - beta1) g,   v' = beta2 v + (1 - beta2) g^2
 *   theta' = theta - lr (m' / (1 - beta1^t)) / (sqrt(v' / (1 - beta2^t)) + delta)
 * for update number t >= 1, g_hat[k] = sum_j coef[j] z_j[k] (j order).  All
 * arithmetic in fp64; theta', m', v' rounded once to fp32.  Coordinates as
 * in oracle_apply_update (ks / nk); ghat (may be NULL) receives g_hat. */
void oracle_apply_adam(const oracle_cfg *c, const float *theta, const float *m, const float *v, int64_t t,
                       uint64_t seed, uint64_t step, float lr, const double *coef, double beta1,
                       double beta2, double delta, double lambda, const int64_t *ks, int64_t nk,
                       float *theta_out, float *m_out, float *v_out, double *ghat) {
  const int P = total_dirs(c);
  const int64_t n = ks ? nk : oracle_param_count(c);
  const double bc1 = 1.0 - pow(beta1, (double)t), bc2 = 1.0 - pow(beta2, (double)t);
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) {
    const int64_t k = ks ? ks[i] : i;
    if (!coord_perturbed(c, k)) {          /* masked: theta and both moments stay */
      theta_out[i] = theta[k];
      m_out[i] = m[k];
      v_out[i] = v[k];
      if (ghat) ghat[i] = 0.0;
      continue;
    }
    double gh = 0.0;
    for (int j = 0; j < P; ++j) {
      float z[4];
      probe_quad(law_of(c, k & ~(int64_t)3), seed, step, (uint32_t)j, (uint64_t)k >> 2, z);
      gh += coef[j] * (double)z[k & 3];
    }
    const double th = (double)theta[k];
    const double g = gh + lambda * th;
    const double m1 = beta1 * (double)m[k] + (1.0 - beta1) * g;
    const double v1 = beta2 * (double)v[k] + (1.0 - beta2) * g * g;
    theta_out[i] = (float)(th - (double)lr * (m1 / bc1) / (sqrt(v1 / bc2) + delta));
    m_out[i] = (float)m1;
    v_out[i] = (float)v1;
    if (ghat) ghat[i] = gh;
  }
}

/* One SPSA step for all experts, accumulated over A = accum independently
 * sampled batches (Appendix E): direction j of the D = A P directions is
 * evaluated on batch j / P, and the estimate averages all D directions,
 *   g_hat = (1/A) sum_a (1/P) sum_{j in batch a} ... = (1/D) sum_j ...
 * Each expert has its own perturbation radius eps[e] and learning rate
 * lr[e] (the paper's per-expert schedule, Section 4).
 *   theta   [N][d]   fp32, read only
 *   seeds   [N]      per-expert Philox stream seeds
 *   eps, lr [N]
 *   bytes   [A][N][B][T]
 *   losses  [N][D][2] out: [e][j][0] = L(theta_e + eps_e z), [1] = L(theta_e - eps_e z)
 *   coef    [N][D]    out (may be NULL): the coefficient applied to z_{e,j}
 *   theta_out [N][d]  out
 *   ghat    [N][d]    out (may be NULL): the estimate, fp64
 * Coefficients: independent losses c_{e,j} = (L_{e,j,+} - L_{e,j,-}) /
 * (2 eps_e D) (Section 4, Eq. main-spsa per expert).  Summed loss (Appendix
 * J): the joint direction perturbs expert e by eps_e z_{e,j}, the shared loss
 * F = sum_e L_e changes by dF_j = sum_e (L_{e,j,+} - L_{e,j,-}), and Eq.
 * main-spsa applied to F gives expert e the coefficient dF_j / (2 eps_e D)
 * (one scalar loss difference shared by every expert, divided by the radius
 * along that expert's coordinates).
 * Returns 0, or -1 on an invalid configuration. */
int oracle_spsa_step_rates(const oracle_cfg *c, const float *theta, const uint64_t *seeds, uint64_t step,
                           const float *eps, const float *lr, const uint8_t *bytes, float *losses, double *coef,
                           float *theta_out, double *ghat) {
  const int N = c->n_experts, P = total_dirs(c), Pb = c->n_pairs;
  if (N < 1 || Pb < 1 || c->n_layers < 1 || c->embed < 1 || c->hidden < 1 || c->batch < 1 ||
      c->seq_len < 2 || c->probe < 0 || c->probe > 2 || c->accum < 0 || c->arch < 0 || c->arch > 2 ||
      c->perturb_mask > 7u || (c->arch == 1 && (c->embed != c->hidden || !c->tied_head)) ||
      (c->arch == 2 && (c->embed % 4 != 0 || !c->tied_head)))
    return -1;
  const int64_t d = oracle_param_count(c);
  const size_t bstride = (size_t)c->batch * c->seq_len;
  double *L = (double *)malloc(sizeof(double) * (size_t)N * P * 2);
  /* 1-4: perturbed forwards, each on its expert's own batch (batch j / Pb of
   * the update for direction j). */
  for (int e = 0; e < N; ++e) {
    oracle_cfg ce = *c;                      /* expert e's tied head (arch 1, 2) */
    if (c->tied_head) ce.tied_head = c->tied_head + e * c->head_stride;
    for (int j = 0; j < P; ++j)
      for (int s = 0; s < 2; ++s)
        L[((size_t)e * P + j) * 2 + s] =
            oracle_perturbed_loss(&ce, theta + (size_t)e * d, seeds[e], step, (uint32_t)j,
                                  s == 0 ? +1 : -1, eps[e],
                                  bytes + ((size_t)(j / Pb) * N + e) * bstride);
  }
  /* 5: coefficients. */
  double *cf = (double *)malloc(sizeof(double) * (size_t)N * P);
  for (int e = 0; e < N; ++e)
    for (int j = 0; j < P; ++j) {
      double diff;
      if (c->loss_mode == 1) {
        diff = 0.0;
        for (int e2 = 0; e2 < N; ++e2)
          diff += L[((size_t)e2 * P + j) * 2 + 0] - L[((size_t)e2 * P + j) * 2 + 1];
      } else {
        diff = L[((size_t)e * P + j) * 2 + 0] - L[((size_t)e * P + j) * 2 + 1];
      }
      cf[(size_t)e * P + j] = diff / (2.0 * (double)eps[e] * (double)P);
    }
  /* 6: update. */
  for (int e = 0; e < N; ++e)
    oracle_apply_update(c, theta + (size_t)e * d, seeds[e], step, lr[e], cf + (size_t)e * P, NULL, 0,
                        theta_out + (size_t)e * d, ghat ? ghat + (size_t)e * d : NULL);
  /* 7: outputs. */
  for (size_t i = 0; i < (size_t)N * P * 2; ++i) losses[i] = (float)L[i];
  if (coef)
    for (size_t i = 0; i < (size_t)N * P; ++i) coef[i] = cf[i];
  free(cf);
  free(L);
  return 0;
}

/* The step with one radius and one learning rate for every expert. */
int oracle_spsa_step(const oracle_cfg *c, const float *theta, const uint64_t *seeds, uint64_t step,
                     float eps, float lr, const uint8_t *bytes, float *losses, double *coef,
                     float *theta_out, double *ghat) {
  if (c->n_experts < 1) return -1;
  float *ev = (float *)malloc(sizeof(float) * 2 * (size_t)c->n_experts);
  for (int e = 0; e < c->n_experts; ++e) {
    ev[e] = eps;
    ev[c->n_experts + e] = lr;
  }
  const int rc = oracle_spsa_step_rates(c, theta, seeds, step, ev, ev + c->n_experts, bytes, losses, coef,
                                        theta_out, ghat);
  free(ev);
  return rc;
}

/* Unperturbed mean cross entropy of every expert on its own batch. */
int oracle_eval_loss(const oracle_cfg *c, const float *theta, const uint8_t *bytes, double *loss) {
  const int64_t d = oracle_param_count(c);
  const size_t bstride = (size_t)c->batch * c->seq_len;
  for (int e = 0; e < c->n_experts; ++e) {
    oracle_cfg ce = *c;
    if (c->tied_head) ce.tied_head = c->tied_head + e * c->head_stride;
    loss[e] = oracle_forward_loss(&ce, theta + (size_t)e * d, bytes + (size_t)e * bstride);
  }
  return 0;
}

int oracle_num_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}
