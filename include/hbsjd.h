/*
 * hbsjd.h - C ABI of the MI355X (gfx950) batched speculative-Jacobi rollout.
 *
 * The library replaces token-by-token student rollout in visual on-policy
 * distillation (paper Sec. 3.1, Eq. 2: the student generates the suffix
 * x_{k+1..T} after a real prefix x_{1..k}). Each image keeps its own committed
 * cursor and window of W draft tokens (Sec. 4.2, "Independent rollout states");
 * all images are verified together in one batched decoder forward over per-image
 * positions and KV locations (Sec. 4.2, "Batched verification"); the
 * probabilistic rule of Eq. 5 (accept with min(1, p/q), otherwise resample from
 * [p - q]_+) or the greedy rule of Eq. 4 commits a variable number of tokens per
 * image (Sec. 4.2, "Independent progress"); and each round runs either the full
 * physical batch or only the active images, Full iff A > gamma (Sec. 4.3, Eq. 6).
 *
 * Conventions used by every call:
 *  - Image tokens sit at sequence positions 1..T (T = grid^2); the class token
 *    sits at position 0. Token arrays are row-major [batch][T]; entry t-1 of a
 *    row is the token at position t.
 *  - "device" pointers are HIP device memory of the GPU the context was created
 *    on; "host" pointers are ordinary host memory. The caller owns every buffer
 *    it passes in; the library never frees or keeps them after the call returns.
 *  - Work is ordered on the context's stream. Calls that return results
 *    (hbsjd_rollout, hbsjd_round, hbsjd_get_state, hbsjd_forward,
 *    hbsjd_verify_probs, hbsjd_philox) block until those results are written.
 *  - A context is used by one host thread at a time.
 *  - Every call returns a status. On any status other than HBSJD_OK,
 *    hbsjd_last_error() (per host thread) describes the failure. HBSJD_EINVAL
 *    is returned before any device work is queued. HBSJD_EHIP and
 *    HBSJD_EINTERNAL poison the context: later calls on it return HBSJD_ESTATE.
 */
#ifndef HBSJD_H_
#define HBSJD_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum hbsjd_status {
    HBSJD_OK = 0,
    HBSJD_EINVAL = 1,     /* bad argument; nothing was queued */
    HBSJD_ENOMEM = 2,     /* device allocation failed or exceeds the KV budget */
    HBSJD_EHIP = 3,       /* a HIP runtime call failed */
    HBSJD_ESTATE = 4,     /* call out of order, or the context is poisoned */
    HBSJD_EINTERNAL = 5   /* a device-side invariant check failed */
} hbsjd_status;

typedef enum hbsjd_dtype {
    HBSJD_DTYPE_F32 = 0,  /* fp32 weights, activations and KV cache */
    /* bf16 weights (rounded to nearest-even on load), held on the GPU as fp16
     * times a power-of-two scale per matrix, exact for every weight down to
     * 2^-31 of its matrix's largest magnitude; fp16 MFMA operands, activations
     * and KV cache (the bf16 operand width and rate, three more mantissa bits);
     * fp32 embeddings, residual stream, accumulation and sampling */
    HBSJD_DTYPE_BF16 = 1
} hbsjd_dtype;

typedef enum hbsjd_exec_mode {
    HBSJD_EXEC_AUTO = 0,     /* per round: Full iff A > gamma (Sec. 4.3, Eq. 6) */
    HBSJD_EXEC_FULL = 1,     /* every round processes all images, finished ones discarded */
    HBSJD_EXEC_COMPACT = 2   /* every round processes only the active images */
} hbsjd_exec_mode;

typedef enum hbsjd_verify_mode {
    HBSJD_VERIFY_PROB = 0,      /* Sec. 4.2, Eq. 5 */
    HBSJD_VERIFY_GREEDY = 1,    /* Sec. 4.2, Eq. 4 */
    /* The cached autoregressive baseline the paper compares against (Sec. 5,
     * Tables 1-5): `window` and `history` are ignored; the prefill covers
     * positions 0..k_b-1 and every round forwards one row per image (its last
     * committed token, or the class token, at position n_b) and commits one
     * token drawn from that row's distribution with u_draft(b, n_b + 1)
     * (Eq. 1). Tokens equal those of HBSJD_VERIFY_PROB with W = 1. */
    HBSJD_VERIFY_AR = 2,
    HBSJD_VERIFY_AR_GREEDY = 3  /* the same, committing the argmax (lowest index on ties) */
} hbsjd_verify_mode;

/*
 * How images move through their windows (Sec. 4.1, "From Single-Sequence to
 * Batched SJD"; Fig. 2; Table 2).
 */
typedef enum hbsjd_progress {
    /* HB-SJD: every image keeps its own cursor and window and advances by its
     * own accepted count each round */
    HBSJD_PROGRESS_INDEPENDENT = 0,
    /* The Batch-Synchronous SJD ablation: window w of image b ends at
     * min(k_b + (w+1) W, T); an image never verifies past its window's end,
     * and one that has reached it waits (its row 0 is still forwarded and its
     * first draft re-drawn from it; it commits nothing and records count 0)
     * until every active image has reached its own, after which the whole
     * batch moves to window w+1. The output distribution is unchanged; the
     * verification rounds grow. Ignored by the AR modes. */
    HBSJD_PROGRESS_SYNC = 1
} hbsjd_progress;

/*
 * The student: a class-conditional LlamaGen-style decoder (Sec. 3.1, Eq. 1;
 * the paper's students are LlamaGen-B and -L). Pre-norm blocks of RMSNorm ->
 * QKV -> 2D RoPE -> causal attention -> O projection + residual -> RMSNorm ->
 * SwiGLU MLP + residual; final RMSNorm and lm_head (optional bias).
 * d_model must be a multiple of n_heads, head_dim = d_model / n_heads a
 * multiple of 4; vocab a multiple of 4 and <= 16384. bf16 needs head_dim == 64
 * and d_model, mlp_hidden and vocab multiples of 64; fp32 needs head_dim <= 64
 * and grid^2 <= 959. Class index n_classes is the null class used by
 * classifier-free guidance.
 */
typedef struct hbsjd_model_desc {
    int32_t n_layers;
    int32_t d_model;
    int32_t n_heads;
    int32_t mlp_hidden;
    int32_t vocab;
    int32_t n_classes;
    int32_t grid;          /* image tokens T = grid * grid */
    int32_t dtype;         /* hbsjd_dtype */
    int32_t has_lm_bias;
    float rms_eps;         /* e.g. 1e-5 */
    float rope_base;       /* e.g. 10000 */
} hbsjd_model_desc;

typedef struct hbsjd_ctx hbsjd_ctx;

/*
 * Create a context on the current HIP device. `stream` is a hipStream_t (NULL
 * for the default stream) on which all of the context's work is ordered.
 * `max_kv_bytes` caps the KV-cache pool (0 = no cap). Returns EINVAL for an
 * unsupported shape, ENOMEM, EHIP.
 */
hbsjd_status hbsjd_create(const hbsjd_model_desc* model, uint64_t max_kv_bytes, void* stream,
                          hbsjd_ctx** out);

/*
 * Copy the weights to the device (rounding to bf16, nearest-even, for a bf16
 * model). `host_blob` is fp32 host memory in this order, every matrix stored
 * out x in row-major: tok_emb [V x d], cls_emb [(C+1) x d]; per layer g_attn [d],
 * Wqkv [3d x d], Wo [d x d], g_ffn [d], W1 [f x d], W3 [f x d], W2 [d x f]; then
 * g_out [d], W_lm [V x d] and, with has_lm_bias, b_lm [V]. EINVAL when
 * n_floats does not match the model.
 */
hbsjd_status hbsjd_load_weights(hbsjd_ctx* ctx, const float* host_blob, size_t n_floats);

/* Arguments of one rollout (the problem statement of Sec. 3.1, Eq. 2). */
typedef struct hbsjd_rollout_args {
    int32_t batch;                  /* B >= 1 */
    const int32_t* prefix_tokens;   /* device [B][T]; the first prefix_len[b] entries are used */
    const int32_t* prefix_len;      /* host [B]; k_b in [0, T]; image b generates T - k_b tokens */
    const int32_t* class_labels;    /* host [B]; in [0, n_classes) */
    const float* temperature;       /* host [B]; finite, > 0 */
    int32_t window;                 /* W in [1, 64], Jacobi window (Sec. 4.2); ignored by the AR modes */
    int32_t history;                /* H >= 1, history offset of the draft fill (Sec. 4.2) */
    int32_t top_k;                  /* 0 = off; otherwise keep entries >= the k-th largest */
    float cfg_scale;                /* 0 = no guidance; else l_u + s (l_c - l_u) (Sec. 4.2) */
    uint64_t seed;                  /* Philox key */
    int32_t verify_mode;            /* hbsjd_verify_mode */
    int32_t exec_mode;              /* hbsjd_exec_mode */
    int32_t gamma;                  /* AUTO threshold; -1 = the context's calibrated value */
    int32_t max_rounds;             /* capacity of `counts`; >= max_b (T - k_b) */
    int32_t progress;               /* hbsjd_progress; 0 = independent (HB-SJD) */
} hbsjd_rollout_args;

/* Results of one rollout; the caller allocates every array. */
typedef struct hbsjd_rollout_out {
    int32_t* tokens;            /* device [B][T]: the prefix, then the generated suffix */
    int32_t* counts;            /* device [max_rounds][B]: tokens committed per round, 0 if
                                   inactive (or waiting at a synchronous window boundary) */
    int32_t* rounds;            /* host [1]: verification rounds run */
    int32_t* active_per_round;  /* host [max_rounds] or NULL: A at the start of each round */
    int32_t* mode_per_round;    /* host [max_rounds] or NULL: 0 Full, 1 Compact */
    int64_t* stats;             /* host [4] or NULL: drafts verified, drafts rejected,
                                   image-rounds, verifier rows processed */
} hbsjd_rollout_out;

/*
 * Run a whole rollout: prefill of [class, x_1..x_k] for every image, first
 * draft from the student, then verification rounds until every image has T
 * tokens. Blocking. The suffix of image b follows the student's AR distribution
 * given its prefix (probabilistic mode) or the greedy AR sequence (greedy
 * mode); Full, Compact and AUTO give identical results. EINVAL (before any
 * device work) for B < 1, W < 1, H < 1, k_b outside [0, T], a label outside
 * [0, C), a temperature that is not finite and positive, top_k < 0,
 * max_rounds < max_b (T - k_b), or a prefix token outside [0, V) (found by a
 * device check before the prefill). ENOMEM, EHIP, EINTERNAL.
 */
hbsjd_status hbsjd_rollout(hbsjd_ctx* ctx, const hbsjd_rollout_args* args,
                           hbsjd_rollout_out* out);

/* Round-level access for tests: prefill + first window (same checks as
   hbsjd_rollout). The state lives in the context until the next begin. */
hbsjd_status hbsjd_rollout_begin(hbsjd_ctx* ctx, const hbsjd_rollout_args* args);

/*
 * One verification round on the state made by hbsjd_rollout_begin, with an
 * explicit execution mode (hbsjd_exec_mode; AUTO uses the begin call's gamma).
 * `counts` host [B] receives the tokens committed this round (0 if inactive);
 * `active` host [1] receives the number of images still active afterwards.
 * ESTATE without a begin.
 */
hbsjd_status hbsjd_round(hbsjd_ctx* ctx, int32_t exec_mode, int32_t* counts, int32_t* active);

/*
 * Export the rollout state to host arrays (any may be NULL): tokens [B][T]
 * (committed tokens, zero past the cursor), cursors [B] (committed count n_b),
 * drafts [B][W] (the draft at window position n_b + 1 + j; -1 past T and once
 * the image is complete) and q_token_prob [B][W], the probability q(z) that
 * each draft's proposal gives it (Sec. 4.2, Eq. 5): for a reused prediction
 * (Sec. 4.2, "Independent rollout states") the p(z) of the verifier row it was
 * drawn from; 1 for a history token (a point-mass proposal) and for every
 * draft in greedy mode; 0 where drafts holds -1. The state is the one after
 * hbsjd_rollout_begin (prefill and first window) or after the last
 * hbsjd_round. ESTATE without a begin.
 */
hbsjd_status hbsjd_get_state(hbsjd_ctx* ctx, int32_t* tokens, int32_t* cursors, int32_t* drafts,
                             float* q_token_prob);

/*
 * Teacher-forced forward of n_seqs sequences [class, x_1..x_len] through the
 * same kernels (the prefill path). tokens: device [n_seqs][T]; lens, labels:
 * host [n_seqs] (label n_classes = null class); logits: device fp32
 * [sum_s (lens[s] + 1)][V], sequence after sequence, positions 0..len. Uses the
 * rollout's KV pool (invalidates a rollout state).
 */
hbsjd_status hbsjd_forward(hbsjd_ctx* ctx, int32_t n_seqs, const int32_t* tokens,
                           const int32_t* lens, const int32_t* labels, float* logits);

/*
 * Teacher scoring of completed rollouts: the distillation loss of Sec. 3.1,
 * Eq. 3 for one batch. `student` and `teacher` are two contexts on the same
 * GPU with loaded weights, the same grid and the same vocabulary (their depth
 * and width may differ). For every image b with k_b < T both models run a
 * teacher-forced forward over [class, x_1 .. x_{T-1}]; with p_S and p_T the
 * plain softmax of each model's conditional logits at position t-1 (no
 * temperature, top-k or guidance), the per-position divergence is
 *   D_biKL = KL(p_S || p_T) / 2 + KL(p_T || p_S) / 2
 * for the generated positions t = k_b+1 .. T.
 *   tokens        device [B][T]: the completed sequences (x_T is never read)
 *   prefix_len    host [B]: k_b in [0, T]
 *   class_labels  host [B]: in [0, min(student, teacher n_classes))
 *   per_position  device [B][T], written: entry t-1 holds D_biKL at position t,
 *                 0 for t <= k_b
 *   loss          device [B], written: the mean of image b's entries over
 *                 t = k_b+1 .. T (Eq. 3's inner average), 0 when k_b = T
 * Blocking. The logits live in library-owned scratch of each context
 * ((T - k_b) summed over images, times vocab, fp32). Replaces any rollout
 * state of both contexts (as hbsjd_forward does). EINVAL for B < 1, NULL
 * buffers, one context passed twice, mismatched grid or vocabulary, k_b or a
 * label out of range, or a token of x_1 .. x_{T-1} outside [0, vocab); ESTATE
 * without weights; ENOMEM; EHIP.
 */
hbsjd_status hbsjd_score_bikl(hbsjd_ctx* student, hbsjd_ctx* teacher, int32_t B,
                              const int32_t* tokens, const int32_t* prefix_len,
                              const int32_t* class_labels, float* per_position, float* loss);

/*
 * The scoring kernel on caller-supplied rows, for testing: out[r] =
 * D_biKL(softmax(logits_s[r]), softmax(logits_t[r])) (Sec. 3.1, Eq. 3). All
 * pointers are device memory; logits_s and logits_t fp32 [rows][V], out fp32
 * [rows]. V must be a multiple of 4 in [4, 16384]. `stream` may be NULL.
 * Blocking. EINVAL for bad sizes or NULL buffers.
 */
hbsjd_status hbsjd_bikl_rows(const float* logits_s, const float* logits_t, int64_t rows,
                             int32_t V, float* out, void* stream);

/*
 * The distribution transform of the verifier rows (Sec. 4.2: the target p and
 * the reused proposals q are full-vocabulary distributions; guided logits under
 * CFG, "Independent progress") on caller-supplied logits, with the draw each
 * rollout row makes, for testing and for sampling outside a rollout. Per row r:
 *   l = logits[r][0]                       (cfg = 1)
 *   l = lu + cfg_scale (lc - lu)           (cfg = 2: lc = logits[r][0], lu = logits[r][1])
 *   y = l / temperature[r]; with 0 < top_k < V, entries below the top_k-th
 *   largest y (counting ties) are dropped, ties with it kept; p = softmax over
 *   the kept entries, its normaliser summed sequentially inside 64-entry chunks
 *   and then over the chunk totals.
 * Outputs: p [rows][V]; argmax [rows], the first index of the largest l;
 * draw [rows], the inverse-CDF draw from p (same association: the first entry
 * whose chunk prefix plus in-chunk prefix exceeds u * sum p, else the last
 * positive entry) with u = u_draft of Philox key `seed`, counter
 * (r, position[r], 0, 0), position clamped to [0, 2^30].
 * All pointers are device memory: logits fp32 [rows][cfg][V]; temperature fp32
 * [rows] (finite and > 0; not checked); position int32 [rows]; p fp32
 * [rows][V], which may be the logits buffer only when cfg = 1. Blocking.
 * EINVAL before any device work for rows < 1, V not a multiple of 4 in
 * [4, 16384], cfg not 1 or 2, a non-finite cfg_scale with cfg = 2, top_k < 0,
 * a NULL buffer or p aliasing logits with cfg = 2; EINVAL after the transform
 * when a logit is NaN (outputs then undefined); ENOMEM for its scratch (the
 * per-row metadata, 8 bytes per row plus 64); EHIP.
 */
hbsjd_status hbsjd_transform_rows(int32_t rows, int32_t V, const float* logits, int32_t cfg,
                                  float cfg_scale, const float* temperature, int32_t top_k,
                                  uint64_t seed, const int32_t* position, float* p,
                                  int32_t* argmax, int32_t* draw, void* stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc):
 * hbsjd_transform_rows with the same arguments, results and errors, whose
 * per-row metadata lives in a fixed library-owned device array (8 bytes per
 * row plus 64; each GPU the library runs on keeps its copy until the process
 * ends) instead of an allocation per call. It allocates and frees nothing.
 * rows <= HBSJD_NOALLOC_MAX_ROWS, EINVAL beyond. Every call on one GPU uses
 * that GPU's one array: calls that overlap on the same GPU (from several host
 * threads, or queued on several streams without ordering between them) race
 * and give undefined results.
 */
#define HBSJD_NOALLOC_MAX_ROWS 65536
hbsjd_status hbsjd_transform_rows_noalloc(int32_t rows, int32_t V, const float* logits,
                                          int32_t cfg, float cfg_scale, const float* temperature,
                                          int32_t top_k, uint64_t seed, const int32_t* position,
                                          float* p, int32_t* argmax, int32_t* draw, void* stream);

/*
 * The verification kernel (Sec. 4.2, Eq. 5) on caller-supplied rows, for
 * testing; the acceptance test and the replacement draw are the rollout's own
 * code. All pointers are device memory: p and q fp32 [B][W][V] (target and
 * proposal row of draft j), drafts [B][W], u_acc [B][W], u_res [B]. Draft j is
 * accepted iff p_j(z) >= q_j(z) or u_acc < p_j(z) / q_j(z); at the first
 * rejection the replacement is drawn with u_res from [p_j - q_j]_+ (from p_j when
 * that is all zero in fp32). Outputs: counts [B] (accepted drafts plus the
 * replacement) and tokens [B][W] (-1 past the count). V a multiple of 4 in
 * [4, 16384] (EINVAL otherwise). Drafts must lie in [0, V); an image with a
 * draft outside it gets count 0 and no tokens. `stream` may be NULL.
 */
hbsjd_status hbsjd_verify_probs(int32_t B, int32_t W, int32_t V, const float* p, const float* q,
                                const int32_t* drafts, const float* u_acc, const float* u_res,
                                int32_t* counts, int32_t* tokens, void* stream);

/*
 * Philox4x32-10 as the rollout uses it, for testing: key = seed, counter =
 * (b, t, 0, 0) for each of the n pairs in `bt` (device uint32 [n][2]); writes
 * device uint32 [n][4]. `stream` may be NULL.
 */
hbsjd_status hbsjd_philox(uint64_t seed, int32_t n, const uint32_t* bt, uint32_t* out,
                          void* stream);

/*
 * Measurement aid, not an operation of the method: a kernel that keeps the
 * matrix cores busy for its whole run, for reading the MFMA counters against a
 * known duty cycle and for the sustained MFMA rate. `workgroups` workgroups of
 * four wavefronts each issue iters x 8 independent v_mfma_f32_16x16x32_f16
 * (16384 flops each) back to back with no memory traffic, so one launch does
 * workgroups x 4 x iters x 8 x 16384 flops. sink must point to 1 KB of
 * writable device memory; the kernel writes it only if its sums take a value
 * they cannot take. Asynchronous on `stream` (a hipStream_t, NULL = the null
 * stream). Errors: EINVAL (workgroups < 1, iters < 1, sink NULL), EHIP.
 */
hbsjd_status hbsjd_mfma_probe(int32_t workgroups, int32_t iters, float* sink, void* stream);

/*
 * Hardware calibration of the Full/Compact threshold (Sec. 4.3, Eq. 6): a
 * data-independent latency test. On synthetic state (`batch` images halfway
 * through an all-zero prefix of class 0, window `window`, no guidance) it
 * times the verifier forward in Full and in Compact mode with A = 1, 2, 4, ...
 * (below batch) images active, and returns the largest A at which Compact is
 * no slower (within 2% of Full, the timing noise); with every image active
 * the two modes run the same rows, so gamma = batch when Compact was no
 * slower at the largest A timed. The context keeps it as the gamma of
 * rollouts that pass gamma = -1.
 * Rollout outputs never depend on gamma. Needs loaded weights; clears any
 * round-API state (a following hbsjd_round returns HBSJD_ESTATE). Errors:
 * EINVAL (batch < 1, window outside [1, 64], gamma NULL), ESTATE (no
 * weights), ENOMEM, EHIP.
 */
hbsjd_status hbsjd_calibrate_gamma(hbsjd_ctx* ctx, int32_t batch, int32_t window,
                                   int32_t* gamma);

/*
 * Per-kernel timing on the context's stream, for measurement. Kernel classes
 * of one verifier round (and of the prefill, which runs the same kernels).
 */
typedef enum hbsjd_kernel {
    HBSJD_K_SETUP = 0,      /* active compaction, mode choice, row assembly */
    HBSJD_K_EMBED = 1,      /* embedding gather + first RMSNorm */
    HBSJD_K_QKV = 2,        /* QKV GEMM + 2D RoPE + paged KV append */
    HBSJD_K_ATTN = 3,       /* causal attention over the paged cache */
    HBSJD_K_OPROJ = 4,      /* O projection + residual */
    HBSJD_K_NORM = 5,       /* RMSNorm (mid-layer, next layer, final) */
    HBSJD_K_W13 = 6,        /* W1|W3 GEMM + SwiGLU */
    HBSJD_K_W2 = 7,         /* W2 GEMM + residual */
    HBSJD_K_LMHEAD = 8,     /* lm_head GEMM (+ bias) */
    HBSJD_K_TRANSFORM = 9,  /* CFG, temperature, top-k, softmax, chunk prefix */
    HBSJD_K_VERIFY = 10,    /* verification, commit, window refresh */
    HBSJD_K_BIKL = 11,      /* teacher scoring: per-position bidirectional KL (Eq. 3) */
    HBSJD_K_COUNT = 12
} hbsjd_kernel;

/*
 * Start timing: from now on launches of the classes whose bit is set in
 * `class_mask` (bit k = hbsjd_kernel k) are bracketed by HIP events on the
 * context's stream, every launch or one in hbsjd_profile_sample's interval;
 * counters restart at zero. class_mask 0 stops timing. Timing adds event
 * records to the bracketed launches and does not change results.
 */
hbsjd_status hbsjd_profile_start(hbsjd_ctx* ctx, uint32_t class_mask);

/*
 * Time one launch in `every` of each timed class. hbsjd_profile_start counts
 * each class's launches from zero; launch i is bracketed by events when
 * i % every == 0 and runs unbracketed otherwise, without the events' queue
 * cost (a few microseconds per bracketed launch). hbsjd_profile_read then
 * reports the bracketed launches only. every >= 1 (1, the default, brackets
 * every launch); EINVAL otherwise. Takes effect at once and lasts until the
 * next call.
 */
hbsjd_status hbsjd_profile_sample(hbsjd_ctx* ctx, int32_t every);

/*
 * Read the accumulated timing (synchronises the stream): host arrays of
 * HBSJD_K_COUNT entries, total milliseconds and launch counts per class; either
 * may be NULL.
 */
hbsjd_status hbsjd_profile_read(hbsjd_ctx* ctx, double* total_ms, int64_t* launches);

/* Release the context and its device memory (NULL is ignored). */
void hbsjd_destroy(hbsjd_ctx* ctx);

/* Description of the last failure on this host thread ("" if none). */
const char* hbsjd_last_error(void);

/* Library version string. */
const char* hbsjd_version(void);

#ifdef __cplusplus
}
#endif

#endif /* HBSJD_H_ */
