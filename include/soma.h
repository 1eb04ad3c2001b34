/*
 * soma.h -- C ABI of the MI355X (gfx950) SOMA SPSA hot path.
 *
 * SOMA (arXiv 2609.37899) trains an ensemble of N byte-level LSTM experts
 * with zero-order SPSA.  One step of the method, for every expert e:
 *
 *   1. draw P directions z_{e,j} over all d parameters of e (Gaussian, or
 *      the paper's sparse or dense Rademacher law: soma_config.probe);
 *   2. evaluate the antithetic losses L_{e,j,+-} = L_e(theta_e +- eps z_{e,j})
 *      on the expert's own batch, all directions and both signs sharing it
 *      (Section 4; Appendix E, Eq. localspsa);
 *   3. form the coefficients c_{e,j} = (L_{e,j,+} - L_{e,j,-}) / (2 eps P)
 *      (Section 4, Eq. main-spsa), or in SUMMED mode, from the one shared
 *      loss difference dF_j = sum_e (L_{e,j,+} - L_{e,j,-}),
 *      c_{e,j} = dF_j / (2 eps P) for every expert (Appendix J, independent
 *      vs summed losses);
 *   4. apply theta_e <- theta_e - lr * sum_j c_{e,j} z_{e,j}, regenerating
 *      every z_{e,j} from its counter instead of storing it.
 *
 * The default model (soma_config.arch = SOMA_ARCH_LSTM; the paper's own
 * body is SOMA_ARCH_BODY, below; both bias-free) is: byte embedding
 * Emb[256][E] -> L stacked LSTM layers (gate order i, f, g, o; h0 = c0 = 0
 * per sequence) -> linear head Whead[256][H] -> softmax cross entropy over
 * the 256 byte values (Appendix E, L_CE).  A sequence of T bytes gives T-1
 * (input, target) pairs; L is the mean over all B(T-1) targets, in nats.
 *
 * Parameter layout (one expert, fp32, flat, canonical index k):
 *   Emb[256][E]; for l = 1..L: W_l[4H][in_l + H] with rows in gate blocks
 *   i, f, g, o and columns [input | recurrent], in_1 = E, in_l = H;
 *   Whead[256][H].  d = 256 E + sum_l 4H (in_l + H) + 256 H.
 *
 * Probe stream (exact, reproducible bit for bit), Gaussian law: z_{e,j}[k]
 * is element k & 3 of the Gaussian quad for q = k >> 2, obtained from
 *   Philox4x32-10 (Salmon et al., SC'11) with
 *     key     = (lo32(seed_e), hi32(seed_e) ^ hi32(step)),
 *     counter = (lo32(q), j, lo32(step), hi32(q)),
 *   and Box-Muller on the word pairs (w0, w1) -> z[4q], z[4q+1] and
 *   (w2, w3) -> z[4q+2], z[4q+3]:
 *     u1 = ((wa >> 8) + 1) 2^-24, u2 = (wb >> 8) 2^-24,
 *     za = sqrt(-2 ln u1) cos(2 pi u2), zb = sqrt(-2 ln u1) sin(2 pi u2),
 *   where ln, cos and sin are fixed fp32 series evaluations (an atanh series
 *   for ln, Taylor series of sin and cos of (pi/2) r after an exact
 *   quarter-turn reduction) with correctly rounded +, *, /, fma and sqrt.
 * Rademacher laws: coordinate k reads the 2-bit field f at bits 2 (k & 15)
 *   of word (k >> 4) & 3 of the Philox output for the same key and counter
 *   (lo32(b), j, lo32(step), hi32(b)), b = k >> 6.  Sparse (the paper's
 *   training law, Appendix E): z = 0 if f < 2, else (f & 1 ? -1 : +1), i.e.
 *   0 w.p. 1/2 and +-1 w.p. 1/4 each.  Dense (the law of its variance theory,
 *   Section 4 and Appendix F): z = f & 1 ? -1 : +1.
 *   Perturbed weights are fmaf(+-eps, z, theta) (one rounding).
 *
 * Conventions for every entry point:
 *   - Pointers named *_dev are device pointers (HIP), caller owned, and must
 *     stay valid until the work enqueued on `stream` has finished.  Other
 *     pointers are host pointers read before the call returns.
 *   - `stream` is a hipStream_t (NULL = the default stream).  Work is
 *     asynchronous; the caller synchronises.
 *   - The library allocates no device memory: scratch space is the caller's
 *     workspace buffer, sized by soma_workspace_size().
 *   - Return value: SOMA_OK or a negative error code; on error nothing is
 *     enqueued and no output is modified.  soma_last_error() returns a
 *     thread-local description of the last error.
 */
#ifndef SOMA_H_
#define SOMA_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SOMA_VOCAB 256

enum soma_status {
  SOMA_OK = 0,
  SOMA_EINVAL = -1,     /* null pointer, bad scalar (eps <= 0, non-finite lr), bad mode */
  SOMA_ESHAPE = -2,     /* unsupported shape (see soma_config) */
  SOMA_EDEVICE = -3,    /* a HIP call or kernel launch failed */
  SOMA_EWORKSPACE = -4  /* workspace missing, misaligned or too small */
};

enum soma_loss_mode {
  SOMA_LOSS_INDEPENDENT = 0, /* c_{e,j} from expert e's own losses (Section 4) */
  SOMA_LOSS_SUMMED = 1       /* c_j from the summed loss, applied to all experts (Appendix J) */
};

/* Probe laws (soma_config.probe; the stream definitions are above). */
enum soma_probe_law {
  SOMA_PROBE_GAUSSIAN = 0,          /* z ~ N(0, 1) */
  SOMA_PROBE_SPARSE_RADEMACHER = 1, /* 0 w.p. 1/2, +-1 w.p. 1/4 each (Appendix E) */
  SOMA_PROBE_RADEMACHER = 2         /* +-1 w.p. 1/2 each (Section 4; Appendix F) */
};

/* Execution flags (soma_config.flags). */
enum soma_flags {
  /* Run the recurrence as one launch per time step with fp32 matrix
   * products (probes regenerated per step), even where the persistent, the
   * one-block (H = 64) or the split-product per-step kernel applies.  Those
   * form each fp32 product from fp16 parts: x = hi + lo, both rounded toward
   * zero, and a b = a_hi b_lo + a_lo b_hi + a_hi b_hi with fp32
   * accumulation.  For |x| <= 65504 the split's error is at most
   * 2^-21 |x| + 2^-24 (about 21 significant bits from |x| = 2^-3 up, fewer
   * below, where the parts fall into fp16's subnormals), so results agree
   * within that rounding; this path is the fp32 reference.  A perturbed
   * weight outside +-65504, or NaN, aborts the step on the device (losses
   * read NaN, theta and the Adam moments are left untouched); activations
   * are bounded by the cell (|h| < 1).  For SOMA_ARCH_BODY every folded
   * matrix weight must stay within +-256 and every decoder gain within
   * +-4096, which keeps each split operand of the body within +-65504. */
  SOMA_FLAG_PER_STEP_RECURRENCE = 1,
  /* Run the input projections of layers 2..L and the output head as row
   * tiles with fp32 matrix products that regenerate their probes per tile,
   * even where the streaming kernels (probes drawn once per 128 weight rows,
   * weights held in registers, split fp16 products) apply.  Results agree
   * within the split products' rounding. */
  SOMA_FLAG_TILED_WEIGHTS = 2,
  /* Run the persistent recurrence with fp32 h staged by every block of a
   * group, even where the pipelined split exchange applies (four row tiles
   * in flight, h published once in split form and copied into LDS by DMA).
   * Both form the same split products; the exchange adds the gate inputs
   * after them rather than before, so results agree within that rounding. */
  SOMA_FLAG_STAGED_RECURRENCE = 4,
  /* Store each layer's output sequence in fp32 and let the next layer's
   * streaming projection split it while staging it, even where the
   * exchange recurrence stores it pre-split in fragment order for the
   * DMA-staged projection (B = 64, H = 128, 256, 512).  Both split the same
   * fp32 values the same way, so results agree bit for bit. */
  SOMA_FLAG_FP32_SEQUENCE = 8
};

/* Parameter groups that soma_config.perturb_mask names.  A masked group
 * gets neither perturbation nor update: its weights enter every perturbed
 * forward unchanged and keep their values (and Adam moments) through the
 * step.  The paper keeps its decoder/embedding E out of the search and
 * perturbs the body only, which lowers the search dimension (Section 4;
 * Appendix E); for the stacked LSTM the three groups can be left out in any
 * combination.  For SOMA_ARCH_BODY theta is one group (SOMA_PERTURB_LSTM),
 * which the mask must include. */
enum soma_perturb_group {
  SOMA_PERTURB_EMBEDDING = 1,  /* Emb[256][E] */
  SOMA_PERTURB_LSTM = 2,       /* W_1 .. W_L (SOMA_ARCH_BODY: the whole body) */
  SOMA_PERTURB_HEAD = 4,       /* Whead[256][H] */
  SOMA_PERTURB_ALL = 7
};

/* Expert architectures (soma_config.arch). */
enum soma_arch {
  /* The stacked LSTM with a perturbed byte embedding and an untied linear
   * head (the layout above). */
  SOMA_ARCH_LSTM = 0,
  /* The paper's expert body (Section 3; Appendix C, Fig. arch): width
   * d = embed = hidden, D = n_layers pre-norm residual blocks
   *   x <- x + LSTM(LN(x; g1)),  x <- x + W2 GELU(W1 LN(x; g2)),
   * bias-free, with a final f = LN(x; g_f) and logits = f E^T, where the
   * tied matrix E [256][d] embeds the input byte (x_0 = E[byte]) and is set
   * with soma_set_tied_head().  E is not perturbed and not part of theta.
   * LN(x; g) = g (x - mean) / sqrt(var + 1e-5) (biased variance over the d
   * features); GELU(u) = u Phi(u) with the exact normal CDF.  Parameters of
   * one expert, canonical order, per block:
   *   g1[d]; W[4d][2d] (gate rows i, f, g, o; columns [LN input | recurrent]);
   *   g2[d]; W1[4d][d]; W2[d][4d];
   * then g_f[d]: d_e = D (16 d^2 + 2 d) + d (the paper's 16 D d^2 + (2D+1) d).
   * Under the sparse Rademacher law the gains g1, g2 and g_f draw dense
   * +-1 (Appendix E); every other coordinate follows soma_config.probe.
   * Supported: d in {16, 32}, D in {1, 2} (one perturbed body and E fit in
   * one compute unit's LDS); flags must be 0. */
  SOMA_ARCH_BODY = 1,
  /* The body of the paper's wider fixed-size controls (Appendix C, counting
   * rules and Table fixed-parameter-counts; Appendix E): the blocks of
   * SOMA_ARCH_BODY at width d_t = hidden between an input projection from
   * the head width d_E = embed and an output projection back to it,
   *   x_0 = P_in E[byte];  the D blocks;  f = LN(x; g_f);  u = P_out f;
   *   logits = u E^T,
   * with each expert's own tied matrix E [256][d_E] (soma_set_tied_head with
   * a nonzero stride), which the perturbation never touches and only the
   * delta rule updates (soma_head_delta; u is the decoder input).  Parameters
   * of one expert, canonical order (every matrix row a multiple of 4 long,
   * so that a probe quad lies in one row of one matrix):
   *   P_in[d_t][d_E]; per block A[d_t][4 d_t] (LSTM input weights, column
   *   g d_t + u for gate g = i, f, g, o of unit u), R[d_t][4 d_t] (recurrent
   *   weights, same columns), U[d_t][4 d_t] (MLP up), V[d_t][4 d_t] (MLP
   *   down, row = output feature); P_out[d_t][d_E]; then the gains g1, g2
   *   of every block and g_f, d_t each:
   *   d_e = 16 D d_t^2 + (2 D + 1) d_t + 2 d_E d_t.
   * Under the sparse probe law the gains draw dense +-1.  The whole body is
   * one group (SOMA_PERTURB_LSTM).  Supported: d_E = 32, 4 <= d_t <= 512
   * (padded inside to a multiple of 64), batch <= 64, one slot's gate inputs
   * B (T-1) 4 d_p floats under 2^31 bytes; flags must be 0; the recurrence
   * needs a device with cooperative launches (SOMA_EDEVICE otherwise). */
  SOMA_ARCH_WIDE = 2
};

/* Shape of one SPSA step.  Constraints: n_experts, n_layers, n_pairs >= 1;
 * embed and hidden positive multiples of 16 (SOMA_ARCH_WIDE: see there); batch >= 1; seq_len >= 2;
 * accum >= 0; pair_chunk in [0, D] (0 picks a chunk that keeps the workspace
 * under 64 GiB; the step processes its D directions in chunks of this many,
 * which changes memory use but not the result); flags: enum soma_flags.
 *
 * Accumulation (Appendix E): with A = accum > 1 an update averages the
 * estimates of A independently sampled batches, each with its own P =
 * n_pairs directions.  The step then evaluates D = A P directions, direction
 * j (probe stream index j) on batch j / P; bytes are [A][N][B][T], losses
 * [N][D][2], coefficients [N][D] with c = (L+ - L-) / (2 eps D).  With A <= 1,
 * D = P and bytes are [N][B][T]. */
typedef struct soma_config {
  int32_t n_experts;  /* N */
  int32_t n_layers;   /* L */
  int32_t embed;      /* E */
  int32_t hidden;     /* H */
  int32_t batch;      /* B sequences per expert */
  int32_t seq_len;    /* T bytes per sequence */
  int32_t n_pairs;    /* P antithetic directions per expert (2P forwards) */
  int32_t loss_mode;  /* enum soma_loss_mode */
  int32_t pair_chunk; /* directions evaluated per pass; 0 = automatic */
  int32_t flags;      /* enum soma_flags, 0 by default */
  int32_t probe;      /* enum soma_probe_law, 0 (Gaussian) by default */
  int32_t accum;      /* A accumulation batches per update (0 or 1: one batch), see below */
  int32_t arch;       /* enum soma_arch, 0 (stacked LSTM) by default */
  uint32_t perturb_mask; /* enum soma_perturb_group bits of the perturbed and updated
                            groups; 0 means SOMA_PERTURB_ALL */
} soma_config;

typedef struct soma_ctx soma_ctx;

/* d, the number of parameters of one expert (layout above).  Pure. */
int soma_param_count(const soma_config* cfg, int64_t* per_expert);

/* Bytes of device workspace soma_create() needs for this shape.  Pure. */
int soma_workspace_size(const soma_config* cfg, size_t* bytes);

/* Bind a shape to a caller-owned device workspace of at least
 * soma_workspace_size() bytes, 256-byte aligned.  The context is host
 * memory owned by the library until soma_destroy(); one context must not be
 * used by two streams at once (its workspace is shared). */
int soma_create(const soma_config* cfg, void* workspace_dev, size_t workspace_bytes,
                soma_ctx** out);
void soma_destroy(soma_ctx* ctx);

/* One SPSA step (Section 4, Eq. main-spsa; Appendix E, Eq. localspsa, with
 * a plain step theta <- theta - lr g_hat in place of Adam).  This is the
 * soma_spsa_step(experts, seeds, eps, lr, byte_batches) of the method with
 * three choices of form: the experts' parameters are one contiguous [N][d]
 * device array rather than N device pointers, so one launch covers every
 * expert; the seeds are a device array, so a step enqueues no host-to-device
 * copy and can be replayed without host work; and the step counter that keys
 * the probe stream is explicit.
 * Where the shape allows (H <= 704 and a multiple of 64, B <= 64, a device
 * that supports cooperative launches), each layer's recurrence runs as one persistent
 * launch whose blocks synchronise per time step through bounded waits; if a
 * wait ever times out, the step's losses are NaN and theta is left
 * unchanged.
 *   theta_dev  [N][d] fp32, updated in place.  It is written only by the
 *              final update kernel, after every loss of the step exists.
 *   seeds_dev  [N] uint64, the per-expert probe stream seeds.
 *   step       the step counter that keys the probe stream.
 *   eps        perturbation radius, finite and > 0.
 *   lr         learning rate, finite.
 *   bytes_dev  [N][B][T] uint8, expert e's batch (shared by all its
 *              directions and both signs); [A][N][B][T] with accumulation.
 *   losses_dev [N][D][2] fp32 out: [e][j][0] = L(theta_e + eps z_{e,j}),
 *              [e][j][1] = L(theta_e - eps z_{e,j}), mean nats per target.
 * The coefficients of the step stay in the workspace until the next call
 * and can be read with soma_coefficients(). */
int soma_spsa_step(soma_ctx* ctx, float* theta_dev, const uint64_t* seeds_dev, uint64_t step,
                   float eps, float lr, const uint8_t* bytes_dev, float* losses_dev, void* stream);

/* soma_spsa_step for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid allocation):
 * no context and no workspace.  The step's scratch space is a static device
 * array of the library, 32 MiB on each GPU it runs on, held until the
 * process ends; shapes whose workspace for one direction at a time exceeds
 * it return SOMA_ESHAPE (the tiny and small shapes fit: the N = 1, H = 64
 * workload needs 1.3 MB).  The directions run in the largest chunk that fits
 * (or cfg->pair_chunk).  Stacked LSTM only (SOMA_EINVAL for SOMA_ARCH_BODY).
 * Calls share that array on each GPU: calls that overlap on one GPU (two
 * streams, two threads) race and must be serialised by the caller; the
 * coefficients are not kept.  Arguments, results, atomicity and errors
 * otherwise as soma_spsa_step, whose kernels it runs, and the results are
 * the same bit for bit at the same chunk. */
int soma_spsa_step_noalloc(const soma_config* cfg, float* theta_dev, const uint64_t* seeds_dev, uint64_t step,
                           float eps, float lr, const uint8_t* bytes_dev, float* losses_dev, void* stream);

/* Adam hyperparameters of the paper's update (Appendix E, Eq. localspsa;
 * the paper uses beta1 = 0.9, beta2 = 0.999, delta = 1e-8 and coupled weight
 * decay 1e-4).  beta1, beta2 in [0, 1); delta finite and > 0; weight_decay
 * finite. */
typedef struct soma_adam {
  float beta1;
  float beta2;
  float delta;         /* stabiliser added to sqrt(v_hat) */
  float weight_decay;  /* lambda: lambda theta is added to the estimate before the moments */
} soma_adam;

/* One SPSA step with the paper's Adam-style update instead of the plain
 * one (steps 1-3 as soma_spsa_step, then for every coordinate)
 *   g = g_hat + lambda theta,  g_hat = sum_j c_{e,j} z_{e,j} (j order, fp32),
 *   m <- beta1 m + (1 - beta1) g,   v <- beta2 v + (1 - beta2) g^2,
 *   theta <- theta - lr (m / (1 - beta1^t)) / (sqrt(v / (1 - beta2^t)) + delta).
 *   m_dev, v_dev  [N][d] fp32 moment buffers (caller owned, 16-byte aligned,
 *                 zero before the first update), updated in place.
 *   t             the update number, >= 1 (the bias corrections' exponent).
 *   hp            host pointer to the hyperparameters.
 * Other arguments, errors and atomicity as soma_spsa_step: theta, m and v
 * are written only by the final update kernel, and an aborted step leaves
 * all three untouched. */
int soma_spsa_step_adam(soma_ctx* ctx, float* theta_dev, float* m_dev, float* v_dev, int64_t t,
                        const soma_adam* hp, const uint64_t* seeds_dev, uint64_t step, float eps, float lr,
                        const uint8_t* bytes_dev, float* losses_dev, void* stream);

/* The Adam update of soma_spsa_step_adam alone, for given coefficients
 * coef_dev [N][D] fp32 (device). */
int soma_apply_adam(soma_ctx* ctx, float* theta_dev, float* m_dev, float* v_dev, int64_t t,
                    const soma_adam* hp, const uint64_t* seeds_dev, uint64_t step, float lr,
                    const float* coef_dev, void* stream);

/* Per-expert learning rate and perturbation radius under the paper's
 * plateau schedule (Section 4; Table experimental-setup: lr and eps start at
 * 1e-3 and are halved together after 1,000 updates without an improvement of
 * the expert's validation loss by more than 1e-8, never below 1e-5).  The
 * state lives in device memory, [N] entries owned by the caller, so a
 * training loop of steps, evaluations and schedule updates needs no host
 * round trip. */
typedef struct soma_schedule_entry {
  float lr;        /* the expert's current learning rate */
  float eps;       /* the expert's current perturbation radius */
  float best;      /* best validation loss observed (+inf before the first) */
  int32_t since;   /* updates since the last improvement or decay */
} soma_schedule_entry;

typedef struct soma_plateau {
  float factor;      /* decay factor in (0, 1): 0.5 */
  int32_t patience;  /* updates without improvement before a decay, >= 1: 1000 */
  float threshold;   /* an improvement must lower the loss by more than this: 1e-8 */
  float floor;       /* lr and eps are not decayed below this: 1e-5 */
} soma_plateau;

/* Set sched_dev[0..n) to (lr0, eps0, +inf, 0).  eps0 finite and > 0. */
int soma_schedule_init(soma_schedule_entry* sched_dev, int32_t n, float lr0, float eps0, void* stream);

/* One observation of the validation losses val_loss_dev [n] fp32 (device,
 * e.g. from soma_eval_loss), `updates` updates after the previous one: for
 * every expert, if val < best - threshold (compared in fp64) then best = val
 * and since = 0, else since += updates; then if since >= patience, lr and eps
 * become min(x, max(x * factor, floor)) and since = 0.  A NaN loss counts as
 * no improvement. */
int soma_schedule_observe(soma_schedule_entry* sched_dev, int32_t n, const float* val_loss_dev, int32_t updates,
                          const soma_plateau* rule, void* stream);

/* soma_spsa_step_adam with each expert's eps and lr read from its schedule
 * entry, sched_dev [N] (device).  The coefficients use the expert's own
 * radius, c_{e,j} = (L+ - L-) / (2 eps_e P); in SUMMED mode the joint
 * direction moves expert e by eps_e z_{e,j}, and Eq. main-spsa applied to the
 * summed loss gives c_{e,j} = dF_j / (2 eps_e P) with the shared difference
 * dF_j = sum_e' (L_{e',j,+} - L_{e',j,-}).  A step with an entry
 * whose eps is not finite and > 0 or whose lr is not finite is aborted on the
 * device: its losses read NaN and theta, m and v stay untouched. */
int soma_spsa_step_adam_sched(soma_ctx* ctx, float* theta_dev, float* m_dev, float* v_dev, int64_t t,
                              const soma_adam* hp, const uint64_t* seeds_dev, uint64_t step,
                              const soma_schedule_entry* sched_dev, const uint8_t* bytes_dev,
                              float* losses_dev, void* stream);

/* Unperturbed mean cross entropy of every expert on its own batch
 * (Appendix E, L_CE; the expert validation loss of Section 6).
 *   theta_dev [N][d] fp32, bytes_dev [N][B][T] uint8, loss_dev [N] fp32 out.
 * The stacked LSTM runs the step's kernels with radius 0 (every weight
 * formed as fma(+-0, z, theta) = theta; split fp16 products): one direction,
 * both signs, the + sign's sum is the loss.  With soma_config.flags set it
 * runs the reference kernels instead (fp32 products, one launch per time
 * step, tiled weights).  A weight outside the split products' range makes
 * the losses NaN. */
int soma_eval_loss(soma_ctx* ctx, const float* theta_dev, const uint8_t* bytes_dev,
                   float* loss_dev, void* stream);

/* The tied matrix E of an SOMA_ARCH_BODY or SOMA_ARCH_WIDE context
 * (Appendix C): expert e reads E_dev + e * expert_stride, [256][w] fp32
 * row-major with w = d (SOMA_ARCH_BODY) or w = d_E = embed (SOMA_ARCH_WIDE)
 * (device, 16-byte aligned, expert_stride a multiple of 4 floats; 0 = one E
 * shared by every expert, the paper's frozen width-32 head; the wide
 * controls give every expert its own).  The context keeps the pointer, not
 * a copy: the memory must stay valid and unchanged while any step or
 * evaluation that reads it runs.  Every step, evaluation and
 * soma_head_delta() on such a context returns SOMA_EINVAL until it is set;
 * SOMA_EINVAL on an SOMA_ARCH_LSTM context. */
int soma_set_tied_head(soma_ctx* ctx, float* E_dev, int64_t expert_stride);

/* The decoder-path delta rule of an SOMA_ARCH_BODY or SOMA_ARCH_WIDE
 * context (Appendix E, Eq. delta): with the decoder inputs f_{b,t} of the
 * unperturbed body held fixed (f = LN(x; g_f), or u = P_out f for the wide
 * body), for every expert
 *   grad_e = (1 / (B (T-1))) sum_{b,t} (softmax(E_e f_{b,t}) - onehot(y_{b,t+1})) f_{b,t}^T,
 * a [256][w] matrix (w as in soma_set_tied_head); the indirect path through
 * the input embedding and the body is deliberately left out.  The wide
 * controls apply it to every expert's own head (Appendix E).
 *   theta_dev [N][d] fp32, bytes_dev [N][B][T] uint8 (device).
 *   lr        if nonzero, also E_e <- E_e - lr grad_e in place (plain
 *             descent on the rule; each expert must then own its E:
 *             expert_stride != 0 or N = 1).
 *   grad_dev  [N][256][w] fp32 out, or NULL.
 *   loss_dev  [N] fp32 out (the unperturbed mean cross entropy, as
 *             soma_eval_loss), or NULL. */
int soma_head_delta(soma_ctx* ctx, const float* theta_dev, const uint8_t* bytes_dev, float lr, float* grad_dev,
                    float* loss_dev, void* stream);

/* Copy the coefficients c[N][D] (fp32) of the last soma_spsa_step on this
 * context into coef_dev (device-to-device, on `stream`). */
int soma_coefficients(soma_ctx* ctx, float* coef_dev, void* stream);

/* The update of step 4 alone, for given coefficients:
 *   theta_e[k] <- theta_e[k] - lr * sum_{j<P} coef[e][j] z_{e,j}[k]
 * (sum in j order, fp32).  coef_dev [N][D] fp32 (device).  This is the
 * kernel soma_spsa_step ends with; it is exposed so that the update can be
 * checked and reused on its own (e.g. to replay a step from stored losses). */
int soma_apply_update(soma_ctx* ctx, float* theta_dev, const uint64_t* seeds_dev, uint64_t step,
                      float lr, const float* coef_dev, void* stream);

/* The Gaussian probe values z_{seed,step,pair}[k] for k in [k0, k0 + count),
 * written to out_dev [count] fp32 (soma_probe with SOMA_PROBE_GAUSSIAN).
 * k0 + count must not exceed 2^40. */
int soma_gaussian(uint64_t seed, uint64_t step, uint32_t pair, uint64_t k0, uint64_t count,
                  float* out_dev, void* stream);

/* The probe values z_{seed,step,pair}[k] for k in [k0, k0 + count) under
 * probe law `law` (enum soma_probe_law), written to out_dev [count] fp32.
 * k0 + count must not exceed 2^40; an unknown law returns SOMA_EINVAL. */
int soma_probe(int law, uint64_t seed, uint64_t step, uint32_t pair, uint64_t k0, uint64_t count,
               float* out_dev, void* stream);

/* Philox4x32-10 on n (counter, key) pairs: ctr_dev [n][4], key_dev [n][2],
 * out_dev [n][4], all uint32 device arrays. */
int soma_philox(const uint32_t* ctr_dev, const uint32_t* key_dev, uint32_t* out_dev, uint64_t n,
                void* stream);

/* The Box-Muller transform of the probe stream on n word pairs:
 * (za[i], zb[i]) from (wa[i], wb[i]) as defined above.  wa_dev, wb_dev [n]
 * uint32, za_dev, zb_dev [n] fp32, all device arrays. */
int soma_box_muller(const uint32_t* wa_dev, const uint32_t* wb_dev, float* za_dev, float* zb_dev,
                    uint64_t n, void* stream);

/* Variance harness (Appendix estimator-iso): moments of the single-direction
 * estimates X_j = D c_{e,j} z_{e,j} of each expert from the coefficients
 * coef_dev [N][D] of a step taken at fixed weights (lr = 0), probes
 * regenerated from (seeds_dev, step):
 *   out_dev[e][0] = sum_k sum_g (sum_{j in g} X_{j,k})^2 over the consecutive
 *                   groups g of `group` directions (group divides D),
 *   out_dev[e][1] = sum_k (sum_j X_{j,k})^2,
 * fp64, out_dev [N][2] (device).  With G = D / group groups and group means
 * Y_g = (1/group) sum_{j in g} X_j, the trace of their covariance across
 * groups is (out[0] - out[1] / G) / (group^2 (G - 1)), and the relative
 * centered variance of an n_pert = group estimate is R_g = that / ||g||^2
 * (for group = 1: the single-probe covariance).  The summation order of the
 * fp64 partial sums is not fixed (atomic adds). */
int soma_estimator_moments(soma_ctx* ctx, const uint64_t* seeds_dev, uint64_t step, const float* coef_dev,
                           int32_t group, double* out_dev, void* stream);

/* Per-phase device time of the last soma_spsa_step on a context, from HIP
 * events recorded on the step's stream between its kernel launches (off by
 * default; enabling adds one event record per phase boundary).  Times are
 * summed over direction chunks. */
typedef struct soma_phase_times {
  float fold_ms;          /* layer-1 gate inputs per byte value (k_fold; 0 where
                             the H = 64 recurrence forms them in the block) */
  float proj_ms;          /* input projections of layers >= 2 (k_proj_dma from a
                             pre-split sequence, k_proj_stream, or the tiled
                             k_proj) */
  float rec_ms;           /* recurrent time steps of all layers (k_rec_xchg or
                             k_rec_persist or, at H = 64, k_rec_local: one launch per layer and
                             chunk; or k_rec_step, one per time step); for
                             SOMA_ARCH_BODY the whole fused forward (k_body) */
  float head_ms;          /* head + softmax cross entropy (k_head_fused at
                             H <= 128, k_head_stream and k_ce_combine above, or
                             the tiled k_head_ce) */
  float reduce_ms;        /* loss sums and coefficients */
  float update_ms;        /* regenerate-and-update (k_update) */
  int32_t rec_launches;   /* recurrence launches in the step */
  int32_t proj_launches;  /* input-projection launches in the step */
  int32_t xchg_launches;  /* of rec_launches, those of the persistent recurrence
                             with the split exchange (k_rec_xchg) */
} soma_phase_times;

/* Turn phase timing on (enable != 0) or off for later steps on ctx. */
int soma_set_phase_timing(soma_ctx* ctx, int enable);

/* Polls a block of the persistent recurrence makes at one group barrier
 * before it gives up, for later steps on ctx (default 2^20, about a second;
 * 0 restores the default).  A block that gives up sets the step's sticky
 * abort flag, every block that sees it leaves, the launch drains and the
 * step is aborted as an invalid rate is: the losses read NaN and theta (and
 * the Adam moments) are left untouched.  A tiny limit exercises that path;
 * it is not a tuning knob.  Errors: SOMA_EINVAL for a NULL ctx. */
int soma_set_spin_limit(soma_ctx* ctx, uint32_t polls);

/* Wait for the last timed step's events and report its phase times.
 * Returns SOMA_EINVAL if no step ran with timing enabled. */
int soma_get_phase_times(soma_ctx* ctx, soma_phase_times* out);

/* Thread-local description of the last error ("" if none). */
const char* soma_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* SOMA_H_ */
