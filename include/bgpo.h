/*
 * bgpo.h - C ABI of the BGPO masked-diffusion ELBO head for AMD MI355X (gfx950).
 *
 * The library computes, for every response b of a batch and every
 * Monte-Carlo sample j of a sample range, the per-sample ELBO term of a
 * masked diffusion language model and the gradient of Boundary-Guided Policy
 * Optimization's linear lower bound through the LM head:
 *
 *   t_{b,j}      timestep drawn from U(0,1) (Eq. mcs_elbo; one per response and
 *                sample, Algorithm 1), or from the stratified grid (j+u)/n_t
 *   mask         each response token masked independently with probability t
 *                (Section 2.1, forward process; the prompt is never masked)
 *   l_{b,j}      (1/t) * sum over masked positions of log softmax(h W)[target]
 *                (Eq. per_step_loss)
 *   d_{b,j}      l_{b,j} - l_old_{b,j} on the same masked sample (Section 3.1)
 *   g_{b,j}      (1+d) A_b / n_t if A_b >= 0, e^d A_b / n_t if A_b < 0 (Eq. g);
 *                prob->bound selects the variants below
 *   loss        += -loss_scale * g_{b,j}   (Algorithm 1: L_j = -g_j / G)
 *   dX, dW      += gradient of that loss term w.r.t. hidden states and head
 *                weights, accumulated sample by sample (Algorithm 1, gradient
 *                accumulation; the lower bound is a sum, Eq. lower_bound_def)
 *
 * Random numbers come from Philox4x32-10 (Salmon et al., SC'11) keyed by
 * (seed mod 2^32, seed div 2^32):
 *   t:           counter (0, seq, j, 1), word 0; T24 = max(word >> 8, 1);
 *                t = T24 * 2^-24
 *   stratified:  counter (0, seq, 0, 2), word 0; U24 = word >> 8;
 *                T24 = max(floor((j * 2^24 + U24) / n_t), 1)
 *   mask:        position i is masked iff resp_mask[b][i] != 0 and
 *                (word (i mod 4) of counter (i div 4, seq, j, 0)) >> 8 < T24
 * where seq = seq_id_base + b.  Masks therefore depend only on
 * (seed, seq, j, resp_mask), never on the batch split, so a later call with
 * other weights reproduces the same masked samples (needed for d_{b,j}).
 *
 * Conventions for every entry point:
 *   - All array arguments are DEVICE pointers (memory of the current HIP
 *     device), owned by the caller; the problem struct is a HOST pointer.
 *   - Work is enqueued on `stream` (a hipStream_t; NULL = default stream) and
 *     is complete when the stream is synchronised.  No entry point
 *     synchronises the stream, except that a non-NULL `prof` makes the call
 *     wait for its own timing events before returning.
 *   - The library never allocates device memory; scratch space is the
 *     caller's `workspace` of at least bgpo_workspace_size() bytes (256-byte
 *     aligned).  Its size depends on B, L, d, V, the input type and the
 *     workspace budget, never on n_t (except in the retain_samples contrast
 *     mode below).
 *   - Without a timing record a call only enqueues kernels (no allocation,
 *     memory set or copy, no synchronisation), so it can be captured into a
 *     HIP graph and replayed; the graph then reads and writes the buffers
 *     that were passed at capture time.
 *   - Host-detectable errors return a negative bgpo_status before anything is
 *     enqueued; HIP launch errors return BGPO_ERR_HIP.  No C++ exception
 *     crosses the ABI.  Entry points keep no mutable global state (except
 *     the static scratch of bgpo_elbo_bwd_accumulate_noalloc); calls on
 *     different streams must not share a workspace.
 *   - hidden (or x) and W_head are row-major; their element type is
 *     prob->in_dtype: bfloat16 bit patterns (uint16, BGPO_BF16) or float32
 *     (BGPO_F32), which the device rounds to bfloat16 (round to nearest
 *     even) on first read, so an fp32 call gives the same bits as a bf16 call
 *     on the host-rounded inputs.
 *   - The head input of sample j may be its own tensor (sample_stride > 0):
 *     the mask predictor's output depends on the noised sequence y_t of each
 *     sample (p_theta(y | y_t, x), Eq. per_step_loss), and the dX of sample j
 *     is then the gradient that its own backward pass consumes.
 *   - Supported shapes: 1 <= B <= 4096, L >= 1, B*L <= 2^20, d % 64 == 0,
 *     V % 64 == 0, 64 <= d <= 65536, 64 <= V <= 2^20, n_t >= 1,
 *     0 <= j_begin, j_count >= 0, j_begin + j_count <= n_t.  Targets must lie
 *     in [0, V) on every response position.  Other shapes return
 *     BGPO_ERR_UNSUPPORTED.
 */
#ifndef BGPO_H_
#define BGPO_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum bgpo_status {
  BGPO_OK = 0,
  BGPO_ERR_INVALID_ARG = -1,   /* NULL pointer, negative size, bad enum, range outside [0, n_t) */
  BGPO_ERR_WORKSPACE = -2,     /* workspace NULL, misaligned or smaller than bgpo_workspace_size() */
  BGPO_ERR_HIP = -3,           /* a HIP call failed (launch, event) */
  BGPO_ERR_UNSUPPORTED = -4,   /* shape outside the supported set above */
  BGPO_ERR_BUDGET = -5         /* no workspace layout fits prob->ws_budget */
} bgpo_status;

/* Element types of the head inputs (bgpo_problem.in_dtype). */
enum { BGPO_BF16 = 0, BGPO_F32 = 1 };

/* Timestep modes. */
enum { BGPO_T_IID = 0, BGPO_T_STRATIFIED = 1 };

/* Objective modes (bgpo_problem.bound), per response b with d_j = l_j - l_old_j:
 *   BGPO_BOUND_PAPER   Eq. g: the first-order Taylor bound (1 + d_j) A / n_t
 *                      (Lemma 1) for A >= 0, the Jensen bound e^{d_j} A / n_t
 *                      (Lemma 2) for A < 0; the tighter lower bound of the two
 *                      for each sign
 *   BGPO_BOUND_TAYLOR  the Taylor term for every sign (ablation of Table 3)
 *   BGPO_BOUND_JENSEN  the Jensen term for every sign (ablation of Table 3)
 *   BGPO_BOUND_EXACT   the ratio objective exp(B_theta - B_old) A itself
 *                      (Eq. elbo_ratio) with B the n_t-sample ELBO estimates:
 *                      g_j = exp(dbar) A / n_t, dbar = mean_j d_j.  Its
 *                      gradient couples all samples, so bgpo_elbo_bwd_accumulate
 *                      requires the full range (j_begin 0, j_count n_t; else
 *                      BGPO_ERR_INVALID_ARG) and, off-policy, first runs a
 *                      forward pass over every sample to form dbar (memory
 *                      stays constant in n_t; the forward work doubles).
 * On-policy (d == 0) all four give g_j = A / n_t and the same gradient.
 *
 * retain_samples = 1 (exact objective only) computes the same result the way
 * an implementation that keeps all n_t computational graphs does (Section 2.2:
 * the exponential of Eq. elbo_ratio needs every sample before any gradient):
 * every sample's forward runs once and its state (masked rows, log-sum-exp
 * partials, gathered rows, the exponentials of its logits) is kept until the
 * mean log-ratio is known.  bgpo_workspace_size then grows linearly with n_t
 * (about 2.2 GB per sample at B=8, L=512, d=4096, V=126464), which is the
 * memory cost that BGPO's linear bound removes; use it to measure that
 * contrast.  retain_samples = 1 with another bound returns
 * BGPO_ERR_INVALID_ARG.  The retained rows (n_t rounded up to whole units of
 * samples, times B*L rounded up to 256 per sample) must stay below 2^22;
 * larger retained problems return BGPO_ERR_UNSUPPORTED from every entry
 * point, bgpo_workspace_size included.  retain_samples = 1 takes the stored
 * mode only: vocab_chunk and ws_budget must be 0 (else BGPO_ERR_INVALID_ARG). */
enum { BGPO_BOUND_PAPER = 0, BGPO_BOUND_TAYLOR = 1, BGPO_BOUND_JENSEN = 2, BGPO_BOUND_EXACT = 3 };

/* Bits of *status_flags (device int32, OR-ed in, never cleared by the library). */
enum { BGPO_FLAG_NONFINITE = 1 };

typedef struct bgpo_problem {
  int32_t B;            /* responses in the batch */
  int32_t L;            /* padded response length (positions per response) */
  int32_t d;            /* hidden size */
  int32_t V;            /* vocabulary size */
  int32_t n_t;          /* Monte-Carlo samples per response: the 1/n_t of Eq. g */
  int32_t j_begin;      /* first sample index handled by this call */
  int32_t j_count;      /* number of samples handled; any split of [0, n_t) is valid */
  int32_t t_mode;       /* BGPO_T_IID or BGPO_T_STRATIFIED */
  uint64_t seed;        /* Philox key */
  uint32_t seq_id_base; /* global id of response b = 0 (seq = seq_id_base + b) */
  int32_t bound;        /* BGPO_BOUND_*; 0 (the paper's objective) for plain callers */
  int64_t sample_stride;/* elements between the head inputs (and the dX outputs) of
                           consecutive samples of the call's range: sample j reads
                           hidden + (j - j_begin) * sample_stride and accumulates into
                           dX + (j - j_begin) * sample_stride.  0 = one hidden[B, L, d]
                           shared by every sample and one dX.  A multiple of 8, >= 0. */
  float norm_eps;       /* epsilon of the final RMSNorm (the _rmsnorm entry points) */
  int32_t retain_samples;/* 0, or 1 with bound = BGPO_BOUND_EXACT: keep the state of
                           every sample instead of running the forward twice (see
                           below); the workspace then grows with n_t */
  int32_t in_dtype;     /* BGPO_BF16 or BGPO_F32: element type of hidden / x and W_head */
  int32_t vocab_chunk;  /* 0 = backward chosen by ws_budget (below); > 0 = the
                           recompute backward with vocabulary chunks of this many
                           entries (a multiple of 256) */
  uint64_t ws_budget;   /* bytes the workspace may take; 0 = no limit (see below) */
} bgpo_problem;

/* Backward modes and the workspace budget.  Both keep device memory constant
 * in n_t; they trade memory for work:
 *   stored exponentials   the forward GEMM of a unit of samples keeps the
 *                         exponentials of its logits (bf16, rows x V, one
 *                         layout that the dX and dW GEMMs both read) against
 *                         one reference per row, the target logit plus 60 in
 *                         log2 units, so that dZ = s (softmax - onehot) is
 *                         one factor per row times them, except at the
 *                         target: three GEMM passes per sample, a workspace
 *                         of about rows x V x 4 bytes per unit (the two units
 *                         of a dW batch; 24 GB at B=8, L=512, d=4096,
 *                         V=126464 with units of 8 samples).  The dX GEMM
 *                         reads a slab-major bf16 copy of W_head (2 d V
 *                         bytes, re-staged every call).  A row whose target log2-probability
 *                         is below -124 (its exponentials would leave the
 *                         range of bf16 and of the fp32 accumulators) is
 *                         recomputed after the forward from fp32 dot
 *                         products, which is slow but exact in form
 *   recompute             the forward keeps only the per-row log-sum-exp; the
 *                         backward walks the vocabulary in chunks of C
 *                         entries, recomputing that chunk's logits, writing
 *                         its dZ (rows x C) and accumulating dX
 *                         and dW before the next chunk: four GEMM passes per
 *                         sample, nothing of size rows x V is ever stored
 * ws_budget = 0 and vocab_chunk = 0 give the stored mode with units of up to
 * 8 samples within about 32 GB.  A nonzero ws_budget takes that layout if
 * it fits, with the dW batch raised to up to 4 units while the budget allows
 * (fewer read-modify-writes of dW); below it, the stored-mode layout (unit,
 * dW batch, dX split capacity) of least estimated time that fits; if none
 * does, the recompute mode with the unit and chunk width of least estimated
 * extra traffic that fits; if nothing fits, BGPO_ERR_BUDGET.
 * vocab_chunk > 0 forces the recompute mode with that chunk (units sized by
 * ws_budget, or within 32 GB when it is 0).  The smallest layout is the
 * recompute mode with units of one sample and chunks of 256 entries: about
 * 2 d V + B L (8 d + V / 16) bytes (the first term is the transposed head,
 * re-staged every call; the recompute mode reads a bf16 W_head in place,
 * and with BGPO_F32 inputs its slab-major bf16 copy adds another 2 d V).  bgpo_workspace_size reports the size of the chosen layout
 * (at most ws_budget). */

/* Kernel classes reported by the optional timing record. */
enum {
  BGPO_K_TRANSPOSE_W = 0,  /* W[d,V] -> W^T[V,d] staging, once per call */
  BGPO_K_MASK = 1,         /* Philox t and masks + stable compaction */
  BGPO_K_GATHER = 2,       /* masked hidden rows (RMSNorm applied) -> H_c and H_c^T */
  BGPO_K_FWD = 3,          /* fused LM-head GEMM + online log-sum-exp partials (in the
                              backward it also stores the exponentials) */
  BGPO_K_ELL = 4,          /* partial combine, log p, l, d, g, loss, gradient scale */
  BGPO_K_SOFTMAX_GRAD = 5, /* stored exponentials -> dZ = s (softmax - onehot): row factors,
                              target entries, H_c^T scaled, out-of-range rows recomputed */
  BGPO_K_DX = 6,           /* dZ W^T split over the vocabulary */
  BGPO_K_DX_REDUCE = 7,    /* split reduction + scatter-add into dX (+ RMSNorm backward) */
  BGPO_K_DW = 8,           /* H_c^T dZ accumulated into dW */
  BGPO_K_RECOMPUTE = 9,    /* recompute mode: a vocabulary chunk's logits -> its dZ */
  BGPO_K_COUNT = 10
};

/* Optional per-kernel timing (host memory).  When passed to an entry point,
 * elapsed milliseconds (HIP events on `stream`) and launch counts of every
 * kernel class are ADDED to the record, after the call waits for its events. */
typedef struct bgpo_timing {
  double ms[BGPO_K_COUNT];
  int64_t launches[BGPO_K_COUNT];
} bgpo_timing;

/* Library version, (major << 16) | minor. */
int bgpo_version(void);

/* Human-readable name of a bgpo_status value (static string, never NULL). */
const char* bgpo_status_string(int status);

/* Bytes of device workspace needed by bgpo_elbo_fwd and
 * bgpo_elbo_bwd_accumulate for `prob` (depends on B, L, d, V, in_dtype,
 * vocab_chunk and ws_budget; never on n_t outside the retain_samples mode).
 * Writes *bytes and returns BGPO_OK, or a negative status (BGPO_ERR_BUDGET if
 * no layout fits ws_budget). Host only. */
int bgpo_workspace_size(const bgpo_problem* prob, size_t* bytes);

/* The layout bgpo_workspace_size measures for `prob` (see the backward
 * modes above): samples per unit, units per dW GEMM (stored mode), capacity of
 * the dX split partials, vocabulary chunk width (0 = stored exponentials), the
 * workspace bytes and whether the layout keeps a slab-major copy of W_head
 * (the default layout and the budget layouts of least estimated time do; a
 * tight budget may trade it for a larger unit).  Returns BGPO_OK or the status of bgpo_workspace_size.
 * Host only. */
typedef struct bgpo_plan_info {
  int32_t samples_per_unit;
  int32_t dw_batch;
  int32_t dx_splits;
  int32_t vocab_chunk;
  uint64_t workspace_bytes;
  int32_t w_copy;       /* 1: the workspace holds the slab-major bf16 copy of W_head
                           that the dX GEMM reads; 0: the dX GEMM reads W_head itself */
} bgpo_plan_info;

int bgpo_workspace_plan(const bgpo_problem* prob, bgpo_plan_info* info);

/* Timestep and mask of every response for ONE sample j (the forward masking
 * process of Section 2.1 and the t draw of Algorithm 1), compacted.
 *   resp_mask  uint8 [B, L]   1 on response positions (prompt/padding 0)
 *   idx        int32 [B*L]    out: masked flat positions b*L + i in ascending
 *                             order in idx[0 .. N), N = sum of n_masked; the
 *                             rest of the array is left untouched
 *   n_masked   int32 [B]      out: masked positions per response
 *   t_out      float [B]      out: t_{b,j} (exact multiple of 2^-24); may be NULL
 * j must lie in [0, n_t); prob->j_begin/j_count are ignored. */
int bgpo_sample_masks(const bgpo_problem* prob, const uint8_t* resp_mask, int32_t j,
                      int32_t* idx, int32_t* n_masked, float* t_out, void* stream);

/* Forward only: l_{b,j} (Eq. per_step_loss) for j in [j_begin, j_begin + j_count).
 *   hidden    bf16 or fp32 [B, L, d]  final hidden states of the response
 *                              positions (in_dtype; 16-byte aligned)
 *   W_head    bf16 or fp32 [d, V]  LM-head weights (V contiguous; in_dtype;
 *                              16-byte aligned)
 *   targets   int32 [B, L]     clean target token y^i of every position
 *   resp_mask uint8 [B, L]
 *   ell       double [B, n_t]  out: entries (b, j) of the range are written
 *   n_masked  int32  [B, n_t]  out: masked-token counts (same entries)
 *   t_out     float  [B, n_t]  out: timesteps (same entries); may be NULL
 *   prof      host timing record or NULL
 * Deterministic: identical inputs give bit-identical outputs, so `ell` from
 * this call fed back as `ell_old` with the same weights gives d == 0 exactly. */
int bgpo_elbo_fwd(const bgpo_problem* prob, const void* hidden, const void* W_head,
                  const int32_t* targets, const uint8_t* resp_mask,
                  double* ell, int32_t* n_masked, float* t_out,
                  void* workspace, size_t ws_bytes, void* stream, bgpo_timing* prof);

/* Forward + lower-bound term + backward for j in [j_begin, j_begin + j_count),
 * each sample's gradient accumulated before the next sample starts (device
 * memory stays constant in n_t).
 *   adv          float  [B]        advantage A_b of each response (Eq. adv)
 *   ell_old      double [B, n_t]   l under the old policy on the same samples;
 *                                  NULL = on-policy (d == 0 exactly); must not
 *                                  overlap ell or g (BGPO_ERR_INVALID_ARG: the
 *                                  call writes l before it reads l_old)
 *   loss_scale   the 1/G of Algorithm 1 (any finite value)
 *   dX           float  [B, L, d]  += d loss / d hidden (zero rows stay zero
 *                                  for never-masked positions)
 *   dW           float  [d, V]     += d loss / d W_head
 *   ell, g       double [B, n_t]   out: l_{b,j} and g_{b,j} for the range
 *   loss         double [1]        += sum over the range of -loss_scale * g
 *   n_masked     int32  [B, n_t]   out
 *   t_out        float  [B, n_t]   out; may be NULL
 *   status_flags int32  [1]        |= BGPO_FLAG_NONFINITE if a non-finite
 *                                  l, g or gradient scale occurs (values are
 *                                  never clamped); may be NULL
 * The gradients are those of the loss (to be minimised). */
int bgpo_elbo_bwd_accumulate(const bgpo_problem* prob, const void* hidden,
                             const void* W_head, const int32_t* targets,
                             const uint8_t* resp_mask, const float* adv,
                             const double* ell_old, double loss_scale,
                             float* dX, float* dW, double* ell, double* g, double* loss,
                             int32_t* n_masked, float* t_out, int32_t* status_flags,
                             void* workspace, size_t ws_bytes, void* stream,
                             bgpo_timing* prof);

/* bgpo_elbo_bwd_accumulate without a workspace argument, for callers that
 * cannot allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid allocation).  The workspace is a static device
 * array of bgpo_noalloc_scratch_bytes() bytes (128 MiB) inside the library,
 * one per device, held until the process ends; the call allocates nothing.
 * The layout is the one bgpo_workspace_size gives for `prob` with ws_budget
 * set to the scratch size (or to prob->ws_budget if that is smaller), so the
 * results are bit-identical to bgpo_elbo_bwd_accumulate with that budget.
 * Problems whose smallest layout exceeds the scratch return BGPO_ERR_BUDGET
 * before anything is enqueued (at the LLaDA head shape the transposed head
 * alone is 1 GB, so only smaller heads fit); retain_samples = 1 returns
 * BGPO_ERR_INVALID_ARG.  Every call on a device shares that device's array:
 * calls that overlap in time on one device (other streams, other threads)
 * race and must be serialised by the caller.  No state carries over from one
 * call to the next (every kernel writes the scratch it reads). */
int bgpo_elbo_bwd_accumulate_noalloc(const bgpo_problem* prob, const void* hidden,
                                     const void* W_head, const int32_t* targets,
                                     const uint8_t* resp_mask, const float* adv,
                                     const double* ell_old, double loss_scale, float* dX,
                                     float* dW, double* ell, double* g, double* loss,
                                     int32_t* n_masked, float* t_out, int32_t* status_flags,
                                     void* stream);

/* Size in bytes of the static scratch array of bgpo_elbo_bwd_accumulate_noalloc. */
size_t bgpo_noalloc_scratch_bytes(void);

/* The same two calls with the final RMSNorm of the mask predictor fused in
 * front of the LM head: the head input of a position is
 *     h = norm_weight * x / sqrt(mean_i x_i^2 + norm_eps)
 * with x the pre-norm activations ([B, L, d] per sample of in_dtype, laid
 * out as `hidden` above, sample_stride included) and norm_weight fp32 [d]
 * (16-byte aligned).  h is formed in fp32 for the masked positions only and
 * rounded once to bf16 before the head GEMMs.  The backward returns the
 * gradients w.r.t. the norm's input and weight:
 *     dx            float [B, L, d] (+ sample_stride)  += d loss / d x
 *     d_norm_weight float [d]                          += d loss / d norm_weight
 * (dgamma summed over positions in a fixed order: deterministic).  Other
 * arguments, outputs and errors as in bgpo_elbo_fwd / bgpo_elbo_bwd_accumulate;
 * NULL norm_weight or d_norm_weight returns BGPO_ERR_INVALID_ARG. */
int bgpo_elbo_fwd_rmsnorm(const bgpo_problem* prob, const void* x, const float* norm_weight,
                          const void* W_head, const int32_t* targets,
                          const uint8_t* resp_mask, double* ell, int32_t* n_masked, float* t_out,
                          void* workspace, size_t ws_bytes, void* stream, bgpo_timing* prof);

int bgpo_elbo_bwd_accumulate_rmsnorm(const bgpo_problem* prob, const void* x,
                                     const float* norm_weight, const void* W_head,
                                     const int32_t* targets, const uint8_t* resp_mask,
                                     const float* adv, const double* ell_old, double loss_scale,
                                     float* dx, float* d_norm_weight, float* dW, double* ell,
                                     double* g, double* loss, int32_t* n_masked, float* t_out,
                                     int32_t* status_flags, void* workspace, size_t ws_bytes,
                                     void* stream, bgpo_timing* prof);

#ifdef __cplusplus
}
#endif

#endif /* BGPO_H_ */
