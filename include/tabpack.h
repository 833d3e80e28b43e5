/*
 * tabpack.h -- C ABI of the packed-MLP hot path for AMD Instinct MI355X (gfx950).
 *
 * The method (arXiv 2607.05380, "TabPack"): K base MLPs, each with its own
 * sampled hidden width, dropout rate, learning rate and weight decay, are
 * trained in parallel as one "model pack" (Section 3.3) with one "optimizer
 * pack" (Section 3.4), each member on its own base batch with the members'
 * losses summed (Section 3.6); after an epoch every member is scored on
 * validation data and an ensemble is built greedily from the pool of
 * candidates (Section 3.5).
 *
 * Conventions shared by every call
 * --------------------------------
 * - Return value: PACK_OK (0) or a negative PACK_E* code.  The message of the
 *   last failure on the calling thread is available from pack_last_error().
 *   No C++ exception crosses this boundary.
 * - Device pointers are plain HIP device addresses owned by the caller; the
 *   library keeps only non-owning pointers into the workspace bound with
 *   pack_bind() and never allocates device memory.  Host pointers are read or
 *   written synchronously inside the call.
 * - Work is enqueued asynchronously on the given hipStream_t (0 = the null
 *   stream); outputs in device memory are valid once that stream is done.
 * - A handle is not thread-safe; concurrent calls on one handle race.
 * - Row-major storage everywhere.  Feature matrices X are fp32 [N, d_in].
 *   Targets y are fp32 [N] (regression value or binary label 0/1) or int32
 *   [N] class indices for PACK_TASK_MULTI_CE.
 */
#ifndef TABPACK_H
#define TABPACK_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define PACK_OK 0
#define PACK_EINVAL (-1)       /* an argument is out of range or inconsistent */
#define PACK_ESTATE (-2)       /* call not valid in the handle's current state */
#define PACK_EHIP (-3)         /* a HIP runtime call failed */
#define PACK_EUNSUPPORTED (-4) /* a valid request this build does not implement */

enum { PACK_TASK_REG_MSE = 0, PACK_TASK_BIN_BCE = 1, PACK_TASK_MULTI_CE = 2 };
enum { PACK_PREC_BF16 = 0, PACK_PREC_FP32 = 1 };
enum { PACK_PREDICT_MEMBERS = 0, PACK_PREDICT_ENSEMBLE = 1 };
enum { PACK_OPT_ADAMW = 0, PACK_OPT_MUON = 1 };

/* Hyperparameters of one base model (Section 3.7: drawn per member from
 * user-given ranges; one hidden width shared by all hidden layers of the
 * member; App. F lists the number of layers among the sampled parameters).
 * As input (pack_config.members) width, dropout, lr, wd and depth are read;
 * pack_get_hparams() also fills the derived fields. */
typedef struct pack_member_hp {
  int32_t width;           /* hidden width d_k, >= 1 */
  int32_t padded_width;    /* out: d_k rounded up to the quantum q */
  uint32_t drop_threshold; /* out: t_k = floor(p_k * 2^16); an element is kept iff its 16-bit draw >= t_k */
  int32_t depth;           /* hidden Linear-ReLU-Dropout blocks L_k in [1, L]; as input 0 means L */
  double dropout;          /* p_k in [0, 1) */
  double lr;               /* AdamW learning rate, > 0 */
  double wd;               /* AdamW decoupled weight decay, >= 0 */
  double scale;            /* out: inverted-dropout scale s_k = 1 / (1 - p_k) */
  double muon_lr;          /* Muon learning rate of the hidden weights (PACK_OPT_MUON), > 0 */
  int32_t d_emb;           /* periodic embedding size per feature, 8 .. 32 (packs with embeddings) */
  int32_t reserved2;
  double sigma;            /* standard deviation of the embedding frequencies' initial values, > 0 */
} pack_member_hp;

/* Description of a pack.  Ranges are inclusive: width ~ UniformInt[lo, hi],
 * dropout ~ Uniform[lo, hi], lr and wd ~ LogUniform[lo, hi] (Section 3.7;
 * the paper's hyperparameter-space table in App. F lists the same kinds of
 * distributions). */
typedef struct pack_config {
  int32_t K;          /* number of members, 1 .. 65535 */
  int32_t d_in;       /* input features, >= 1 */
  int32_t d_out;      /* outputs: 1 for PACK_TASK_REG_MSE / PACK_TASK_BIN_BCE, classes (2..16) for CE */
  int32_t L;          /* hidden Linear-ReLU-Dropout blocks per member (the maximum with a depth range), 1 .. 8 */
  int32_t B;          /* rows per member per step (base batch), 1 .. 65536 */
  int32_t task;       /* PACK_TASK_* */
  int32_t precision;  /* PACK_PREC_BF16: bf16 MFMA GEMMs, fp32 master weights; PACK_PREC_FP32: fp32 MFMA */
  int32_t width_lo, width_hi;
  int32_t quantum;    /* padding quantum q for widths (multiple of 8); 0 selects 32 */
  int32_t decay_bias; /* 1: weight decay also on biases (torch default), 0: weights only */
  int32_t keep_grads; /* 1: pack_train_step() also stores every gradient for pack_get_grads();
                         0: the hidden-layer weight gradients are consumed by the fused optimizer
                         update without being written out (pack_get_grads() then fails) */
  double dropout_lo, dropout_hi;
  double lr_lo, lr_hi;
  double wd_lo, wd_hi;
  double beta1, beta2, eps; /* AdamW constants, e.g. 0.9, 0.999, 1e-8 */
  uint64_t seed;            /* hyperparameters, initial parameters and dropout masks derive from it */
  const pack_member_hp* members; /* optional [K] explicit hyperparameters; NULL: sample from the ranges */
  int32_t depth_lo, depth_hi;    /* member depth L_k ~ UniformInt[depth_lo, depth_hi], 1 <= lo <= hi <= L;
                                    0, 0: every member has L blocks.  L is the deepest member's depth:
                                    a layer-l launch holds only the members with L_k >= l */
  /* Optimizer pack (Section 3.4; the paper's default trains the main weights of
   * the backbone's linear layers with Muon and every other parameter with
   * AdamW).  PACK_OPT_ADAMW: AdamW everywhere.  PACK_OPT_MUON: the hidden
   * weights W_1..W_Lk take Muon steps (Jordan et al., 2024): momentum buffer
   * B <- mu B + G, direction U = G + mu B (Nesterov) or B, ns_steps
   * Newton-Schulz iterations X <- a X + (b A + c A A) X with A = X X^T from
   * X = U / (||U||_F + 1e-7) (U^T when the true rows exceed the true columns),
   * (a, b, c) = (3.4445, -4.7750, 2.0315), then W <- W (1 - lr_muon wd) -
   * lr_muon max(1, rows/cols)^(1/2) X with the true shape; biases and the head
   * stay on AdamW.  Muon learning rates ~ LogUniform[muon_lr_lo, muon_lr_hi]. */
  int32_t optimizer;             /* PACK_OPT_* */
  int32_t ns_steps;              /* Newton-Schulz iterations, 1 .. 16 (0 selects 5) */
  double muon_lr_lo, muon_lr_hi;
  double muon_momentum;          /* mu in [0, 1) */
  int32_t muon_nesterov;         /* 1: Nesterov direction, 0: the momentum buffer */
  int32_t reserved;
  /* Periodic feature embeddings (App. "Feature Embeddings"): with emb_lo > 0
   * each member maps feature x_i to d_emb values alpha_i * [x_i, cos(w_i x_i +
   * b_i)] + beta_i (w_i, b_i of length d_emb - 1; alpha_i, beta_i of length
   * d_emb), concatenated feature-major into the first layer's d_in * d_emb
   * inputs.  Initial values: w ~ N(0, sigma), b = alpha = beta = 0; trained
   * with AdamW.  d_emb ~ emb_lo + emb_step * UniformInt[0, (emb_hi - emb_lo) /
   * emb_step] (8 <= lo <= hi <= 32, the range App. F samples from), sigma ~
   * LogUniform[sigma_lo, sigma_hi].  Requires B <= 2048.  The member's dense
   * parameter vector then starts with w, b, alpha, beta (row-major
   * [d_in, d_emb - 1] / [d_in, d_emb]); its dense W_1 has the d_in * d_emb
   * columns in that order.  The embedded inputs are never stored: the first
   * layer's GEMMs compute them from the data rows. */
  int32_t emb_lo, emb_hi, emb_step;
  int32_t reserved3;
  double sigma_lo, sigma_hi;
} pack_config;

typedef struct pack_handle pack_handle;

/* Message of the last failed call on this thread ("" if none).  Never NULL. */
const char* pack_last_error(void);

/* Create a pack (host only, allocates no device memory): validate cfg, draw
 * every member's hyperparameters (Section 3.7) unless cfg->members is given,
 * plan the packed layout and generate the initial parameters on the host
 * (torch.nn.Linear's default U(-1/sqrt(fan_in), 1/sqrt(fan_in)) for weights
 * and biases, fan_in = the member's true input width; padding exactly zero).
 * On success *out owns the handle; release it with pack_destroy(). */
int pack_init(const pack_config* cfg, pack_handle** out);

/* Release the handle and its host memory.  The bound workspace stays the
 * caller's.  NULL is accepted. */
int pack_destroy(pack_handle* h);

/* Copy the K members' hyperparameters (inputs and derived fields) to out[K]. */
int pack_get_hparams(const pack_handle* h, pack_member_hp* out);

/* Device workspace (bytes) that pack_bind() needs: parameters, gradients,
 * AdamW moments, bf16 weight shadow, activations and launch tables. */
int pack_workspace_size(const pack_handle* h, size_t* bytes);

/* Bind a caller-owned device workspace of at least pack_workspace_size()
 * bytes (256-byte aligned) and upload the initial parameters; moments and the
 * step counter are reset to zero.  May be called again to move the pack to a
 * new workspace (state is re-initialised from the host copy). */
int pack_bind(pack_handle* h, void* workspace, size_t bytes, hipStream_t stream);

/* Choose which members stay in the pack (Section 3.6, early stopping of base
 * models: a member whose validation score has stopped improving is removed
 * from the pack so that the compute goes to the members still improving).
 *   active  host uint8 [K], 1 = member k is trained and evaluated, 0 = removed
 * A removed member's parameters and AdamW moments are frozen as they are (its
 * getters keep working, its rows of loss_out / pred_out / score_out are no
 * longer written) and its GEMM tiles, head work and optimizer chunks leave the
 * launches.  A member may be re-activated.  All members start active.  With a
 * bound workspace the call re-plans the launches and uploads the tables on
 * `stream` and synchronizes it.  Any subset is valid, including the empty one;
 * training or evaluating an empty pack fails with PACK_ESTATE. */
int pack_set_active(pack_handle* h, const uint8_t* active, hipStream_t stream);

/* One training step of all K members (Sections 3.3, 3.4, 3.6): member k runs
 * forward on its base batch X[idx[k*B + b], :] (b < B) through L blocks
 * H = Dropout_k(ReLU(H W^T + b)) and a linear head, computes its batch-mean
 * loss (MSE, binary CE with logits, or multiclass CE), backpropagates, and
 * takes one AdamW step with its own (lr_k, wd_k).  The pack objective is the
 * sum of the members' losses, so each member receives exactly its own
 * gradient.
 *   X        device fp32 [N, d_in]; y device fp32 [N] or int32 [N] (CE)
 *   idx      device int32 [K, B], every entry in [0, N).  An entry outside
 *            that range is not an error of the call (the step runs
 *            asynchronously): the step reads row 0 in its place and raises
 *            PACK_STATUS_IDX_RANGE, which pack_status() reports.
 *   step     1-based AdamW step t; must be the previous step + 1 (PACK_ESTATE
 *            otherwise).  It is also the dropout counter of this step.
 *   loss_out device fp32 [K]: batch-mean loss of each member before the update
 * Dropout masks: element (r, c) of hidden layer l of member k is kept iff the
 * 16-bit half (r & 1) (0: low bits) of word ((r >> 1) & 3) of
 * Philox4x32-10(counter = (r >> 3, c, (k << 8) | l, step mod 2^32),
 * key = (seed mod 2^32, (seed >> 32) ^ (3 << 28))) is >= t_k. */
int pack_train_step(pack_handle* h, const float* X, const void* y, int64_t N,
                    const int32_t* idx, uint64_t step, float* loss_out, hipStream_t stream);

/* Optional: take the first layer's batch rows straight from the training
 * data (Section 3.3: each member's base batch is a set of rows of X chosen by
 * its indices).  Converts X once into xb (bf16, N rows of d_in rounded up to
 * a multiple of 8, zero-filled) on `stream`; the first layer's forward GEMM of
 * every later pack_train_step() then loads its rows from xb through the batch
 * indices, and so does its weight-gradient GEMM: no gathered copy of the
 * batch is made.  Results are bit-identical to the unbound step.
 *   X      device fp32 [N, d_in], the X every following pack_train_step()
 *          passes (same pointer and N; PACK_EINVAL otherwise); NULL unbinds
 *          (the step then gathers the batch before the first GEMM again)
 *   xb     device buffer owned by the caller, 16-byte aligned, at least
 *          N * round_up(d_in, 8) * 2 bytes (at most 2 GiB), kept until the
 *          data is unbound or the pack destroyed.  The steps read the copy:
 *          after a change of X's contents, call pack_bind_data() again
 * bf16 packs without feature embeddings and with B <= PACK_BIND_DATA_MAX_B
 * only (PACK_EINVAL otherwise). */
#define PACK_BIND_DATA_MAX_B 2048
int pack_bind_data(pack_handle* h, const float* X, int64_t N, void* xb, size_t xb_bytes, hipStream_t stream);

/* Evaluate every active member on validation rows without dropout (Section
 * 3.5 / 3.6: per-epoch validation scoring feeds early stopping and selection).
 *   pred_out  device fp32 [K, Nv]: the per-row value an ensemble averages --
 *             the output (regression), P(class 1) (binary), or the
 *             probability of the true class (multiclass); row k is written
 *             for active members only
 *   score_out device fp64 [K]: RMSE, mean binary CE or mean CE of pred_out
 *             (probabilities clipped to [1e-15, 1 - 1e-15]); non-finite -> +inf;
 *             active members only */
int pack_eval_members(pack_handle* h, const float* Xv, const void* yv, int64_t Nv,
                      float* pred_out, double* score_out, hipStream_t stream);

/* Predictions of the active members on N rows without dropout, as the final
 * ensemble is applied (Section 3.5: the ensemble averages its members'
 * predictions -- class probabilities for classification).
 *   X     device fp32 [N, d_in]
 *   mode  PACK_PREDICT_MEMBERS: out device fp32 [n_active, N, d_out], the
 *         active members in increasing index order;
 *         PACK_PREDICT_ENSEMBLE: out device fp32 [N, d_out], the mean over the
 *         active members (summed in that order in fp64)
 * Values: the output (regression), P(class 1) (binary, d_out = 1) or the
 * softmax probabilities (multiclass).  A pack built from the selected
 * snapshots (explicit hyperparameters, pack_set_params) predicts with the
 * ensemble. */
int pack_predict(pack_handle* h, const float* X, int64_t N, int32_t mode, float* out, hipStream_t stream);

/* Asynchronous error flags raised by the kernels since the last call
 * (PACK_STATUS_* bits; 0: none): waits for `stream`, returns the flags in
 * *flags and clears them.  PACK_STATUS_IDX_RANGE: a pack_train_step() batch
 * index lay outside [0, N). */
#define PACK_STATUS_IDX_RANGE 1u
int pack_status(pack_handle* h, uint32_t* flags, hipStream_t stream);

/* Measurement aid: dst <- src over `bytes` (a multiple of 16; both addresses
 * 16-byte aligned; the ranges must not overlap) with the non-temporal 16-byte
 * loads and stores of the optimizer epilogues, asynchronously on `stream`.  A
 * kernel of known HBM traffic (bytes read + bytes written) against which
 * hardware byte counters and the streaming rate are calibrated.  Allocates
 * nothing. */
int pack_stream_copy(const void* src, void* dst, size_t bytes, hipStream_t stream);

/* Scratch bytes pack_select() needs for C candidates over Nv rows. */
int pack_select_workspace_size(int32_t C, int64_t Nv, size_t* bytes);

/* Greedy ensemble selection (Section 3.5): start from the best single
 * candidate, then repeatedly add -- without replacement -- the candidate whose
 * addition gives the best score of the averaged ensemble; stop at m_ens
 * members or when no addition strictly improves the score.  Ties go to the
 * lowest candidate index; non-finite scores count as +inf and are never
 * picked.  Scores are computed in fp64 with the rule of pack_eval_members.
 *   cand      device fp32 [C, Nv] candidate values (rows of pred_out; for the
 *             online ensemble the K current members followed by the previous
 *             ensemble's frozen members, each a separate candidate)
 *   work      device scratch of pack_select_workspace_size() bytes
 *   sel_out   device int32 [m_ens]: picks in order; n_sel_out device int32 [1];
 *   score_out device fp64 [1]: the final ensemble's score (+inf if empty) */
int pack_select(pack_handle* h, const float* cand, const void* yv, int32_t C, int64_t Nv,
                int32_t m_ens, void* work, size_t work_bytes, int32_t* sel_out,
                int32_t* n_sel_out, double* score_out, hipStream_t stream);

/* pack_select() for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the same selection, with the same arguments and results, but its scratch is
 * a file-scope device array of PACK_SELECT_STATIC_BYTES inside the library
 * (one per GPU, held until the process ends) instead of `work`.  Allocates
 * nothing.  Returns PACK_EINVAL when pack_select_workspace_size(C, Nv)
 * exceeds PACK_SELECT_STATIC_BYTES (e.g. Nv beyond about 500,000 rows).
 * Every call on one GPU shares that GPU's array: calls that overlap on one
 * GPU (from concurrent streams or threads) race and give undefined results. */
#define PACK_SELECT_STATIC_BYTES ((size_t)4 << 20)
int pack_select_static(pack_handle* h, const float* cand, const void* yv, int32_t C, int64_t Nv,
                       int32_t m_ens, int32_t* sel_out, int32_t* n_sel_out, double* score_out,
                       hipStream_t stream);

/* Number of floats in member k's dense parameter vector: for l = 1..L_k the
 * row-major [d_k, fan_in] weight then its [d_k] bias, then the head's
 * [d_out, d_k] weight and [d_out] bias (torch.nn.Linear layout). */
int pack_member_param_count(const pack_handle* h, int32_t member, int64_t* count);

/* Copy member k's parameters to / from a host buffer in the dense layout
 * above.  Before pack_bind() they read/write the host initial values; after
 * it, the device state (synchronous on the null stream). */
int pack_get_params(pack_handle* h, int32_t member, float* host_out);
int pack_set_params(pack_handle* h, int32_t member, const float* host_in);

/* Gradients of the last pack_train_step() (PACK_ESTATE unless the pack was
 * created with keep_grads = 1) and the AdamW moments of member k, dense
 * layout, copied to host buffers (synchronous). */
int pack_get_grads(pack_handle* h, int32_t member, float* host_out);
int pack_get_moments(pack_handle* h, int32_t member, float* m_out, float* v_out);

/* Test hooks.  pack_debug_dropout_mask writes the keep mask (uint8 0/1,
 * [B, d_k]) of hidden layer `layer` (1-based) of member k at `step` to device
 * memory using the same device function as the training epilogue.
 * pack_debug_activation copies the stored post-dropout activation H_layer of
 * member k ([B, d_k] as fp32) of the last forward pass to a host buffer.
 * layer must lie in [1, L_k]. */
int pack_debug_dropout_mask(pack_handle* h, uint64_t step, int32_t layer, int32_t member,
                            uint8_t* dev_out, hipStream_t stream);
int pack_debug_activation(pack_handle* h, int32_t layer, int32_t member, float* host_out);

/* Per-kernel timing of pack_train_step() with HIP events recorded on the
 * stream each kernel runs on, around every launch (measurement aid; it adds
 * two event records per launch).  pack_profile_enable(h, 1) clears and starts
 * recording, 0 stops it.  pack_profile_read() waits for the recorded events
 * and reports, per kernel (one entry per compiled kernel variant, as a
 * profiler names them), the launches seen, their summed duration and the
 * algorithmic work of one launch on the true (unpadded) member shapes: flops,
 * and the bytes an ideal kernel must move to or from HBM (operands read once,
 * outputs written once).  kind names the roofline that bounds the kernel. */
typedef struct pack_kernel_stat {
  char name[64];
  int32_t kind;      /* 0: MFMA-bound (roofline in flops), 1: HBM-bound (roofline in bytes) */
  int32_t launches;
  double total_ms;
  double flops;      /* per launch */
  double bytes;      /* per launch */
  double busy_ms;    /* time during which at least one of its launches ran (launches of concurrent
                        member groups overlap, so this can be less than total_ms) */
} pack_kernel_stat;

int pack_profile_enable(pack_handle* h, int32_t enable);
int pack_profile_read(pack_handle* h, pack_kernel_stat* out, int32_t max, int32_t* n);

#ifdef __cplusplus
}
#endif
#endif /* TABPACK_H */
