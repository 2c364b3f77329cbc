// C-ABI entry points and the host round driver of the batched SJD rollout.
//
// A rollout is: prefill of [class, x_1..x_k] for every image, first draft from
// the student, then rounds of (active compaction + Full/Compact choice, row
// assembly, decoder forward over the paged KV cache, lm_head, distribution
// transform, verification, commit, window refresh) until every image holds T
// tokens (paper Sec. 4.2-4.3). All of a round's launches read their row counts
// from device memory written by the round's own set-up kernel, so the host
// never waits inside a round; it reads the active count of the previous round
// (pinned memory, one round behind) only to know when to stop. Rounds queued
// after the last image finished process zero rows.
#include "hbsjd.h"
#include "common.h"
#include "launch.h"

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

using namespace hbsjd;

namespace hbsjd {
LaunchEvents* launch_events() {
    static thread_local LaunchEvents slot;
    return &slot;
}
}  // namespace hbsjd

namespace {

thread_local std::string g_err;

hbsjd_status fail(hbsjd_status st, const std::string& msg) {
    g_err = msg;
    return st;
}

struct DevBuf {
    void* p = nullptr;
    size_t n = 0;
};

}  // namespace

struct hbsjd_ctx {
    hbsjd_model_desc m{};
    int L = 0, d = 0, H = 0, dh = 0, f = 0, V = 0, C = 0, G = 0, T = 0, nC = 0;
    bool f16 = false;
    size_t esz = 4;
    hipStream_t stream = nullptr;       // the library's own stream (default priority)
    hipStream_t user_stream = nullptr;  // the caller's stream: work starts after its work
    hipEvent_t ev_user = nullptr;
    int device = 0;
    uint64_t max_kv_bytes = 0;
    bool poisoned = false;
    bool weights = false;
    int gamma_cal = -1;

    // weights
    DevBuf wbuf;
    float *tok_emb = nullptr, *cls_emb = nullptr;
    void* w_lm = nullptr;
    float *b_lm = nullptr, *g_out = nullptr;
    // per GEMM matrix: the factor that undoes its storage scale (1 for fp32)
    std::vector<float> s_qkv, s_o, s_13, s_2;
    float s_lm = 1.f;
    std::vector<float*> g_attn, g_ffn;
    std::vector<void*> wqkv, wo, w13, w2;
    DevBuf rope;   // cos then sin, [(T+1)][dh/2] each

    // device buffers, grown on demand
    DevBuf xtok, cursor, drafts, qsrc, labels, temps, plen;
    DevBuf meta, meta_pf, a_hist, mode_hist, stats, counts_own;
    DevBuf row_tok, row_pos, row_kv, row_seq;
    DevBuf seg_seq, seg_row0, seg_nrows, seg_pos0;
    DevBuf slot_img, active_list, pf_slots;
    DevBuf h, hb, qb, ob, act, part;
    DevBuf P[2], amax[2], samp, logits;
    DevBuf seq_row0, seq_img, seq_branch, lm_idx;
    DevBuf ptab, kv;
    DevBuf calib_tok;   // all-zero prefixes of the gamma calibration
    DevBuf seg_pages;   // [segment][max_pages] KV page of each tile (attention's page list)
    DevBuf win_end;     // [B] end of each image's current window (batch-synchronous progress)
    DevBuf qz;          // [B][W] proposal probability of each draft (state export)
    DevBuf score_logits, score_idx, score_k;   // teacher scoring: selected logits rows, their
                                               // output slots, prefix lengths
    int32_t* pin = nullptr;    // pinned host words: active counts of the last two rounds
    hipEvent_t ev[2] = {nullptr, nullptr};

    // rollout state
    bool have_state = false;
    int B = 0, W = 0, Hh = 24, top_k = 0, cfg = 1, greedy = 0, exec_mode = 0, gamma = 0;
    int ar = 0;   // cached-AR baseline rounds (W = 0: one row per image)
    int sync = 0; // batch-synchronous windows instead of independent progress
    hipEvent_t ev_done = nullptr;   // teacher scoring: this context's forward has been queued
    int max_rounds = 0, max_pages = 0, rounds_launched = 0;
    // an upper bound, known on the host, of the images active in the next
    // round (images only ever finish, so a count read a round or two behind
    // bounds it); sizes the kernel choice of the round's products
    int a_bound = 0;
    float cfg_scale = 0.f;
    uint64_t seed = 0;
    int32_t* counts = nullptr;   // device [max_rounds][B]
    long kv_layer_elems = 0;

    // Captured rounds: each a pair of graphs (buffer parity 0 and 1) with the
    // kernels its products were captured with. They are valid while the
    // launch arguments they bake in stay the same (gsig); a pair serves a
    // round whose row bound gives each of its products the same kernels.
    struct RoundGraphs {
        std::vector<GemmPlan> plan;
        int bound = 0;   // the row bound it was captured under
        hipGraphExec_t exec[2] = {nullptr, nullptr};
    };
    std::vector<RoundGraphs> graphs;
    std::vector<uint64_t> gsig;
    bool use_graphs = true;

    // per-kernel-class timing (hbsjd_profile_start / hbsjd_profile_read)
    uint32_t prof_mask = 0;
    int32_t prof_every = 1;                  // one bracketed launch in prof_every
    int64_t prof_seen[HBSJD_K_COUNT] = {};   // launches of each class since profile_start
    std::vector<hipEvent_t> prof_free;
    std::vector<std::pair<int, std::pair<hipEvent_t, hipEvent_t>>> prof_pending;
    double prof_ms[HBSJD_K_COUNT] = {};
    int64_t prof_n[HBSJD_K_COUNT] = {};

    ~hbsjd_ctx();
};

namespace {

hbsjd_status hip_fail(hbsjd_ctx* c, hipError_t e, const char* what) {
    if (c) c->poisoned = true;
    return fail(HBSJD_EHIP, std::string(what) + ": " + hipGetErrorString(e));
}

#define HIPTRY(ctx, x)                                         \
    do {                                                       \
        hipError_t e_ = (x);                                   \
        if (e_ != hipSuccess) return hip_fail((ctx), e_, #x);  \
    } while (0)

hbsjd_status ensure(hbsjd_ctx* c, DevBuf& b, size_t bytes) {
    if (bytes == 0) bytes = 16;
    if (b.n >= bytes) return HBSJD_OK;
    if (b.p) {
        HIPTRY(c, hipStreamSynchronize(c->stream));
        HIPTRY(c, hipFree(b.p));
        b.p = nullptr;
        b.n = 0;
    }
    hipError_t e = hipMalloc(&b.p, bytes);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        b.p = nullptr;
        return fail(HBSJD_ENOMEM, "device allocation of " + std::to_string(bytes) + " bytes failed");
    }
    b.n = bytes;
    return HBSJD_OK;
}

#define TRY(x)                              \
    do {                                    \
        hbsjd_status s_ = (x);              \
        if (s_ != HBSJD_OK) return s_;      \
    } while (0)

template <typename T> T* as(DevBuf& b) { return reinterpret_cast<T*>(b.p); }

void free_buf(DevBuf& b) {
    if (b.p) (void)hipFree(b.p);
    b.p = nullptr;
    b.n = 0;
}

}  // namespace

hbsjd_ctx::~hbsjd_ctx() {
    if (stream) (void)hipStreamSynchronize(stream);
    DevBuf* all[] = {&wbuf, &rope, &xtok, &cursor, &drafts, &qsrc, &labels, &temps, &plen,
                     &meta, &meta_pf, &a_hist, &mode_hist, &stats, &counts_own, &row_tok,
                     &row_pos, &row_kv, &row_seq, &seg_seq, &seg_row0, &seg_nrows, &seg_pos0,
                     &slot_img, &active_list, &pf_slots, &h, &hb, &qb, &ob, &act, &part, &P[0], &P[1],
                     &amax[0], &amax[1], &samp, &logits, &seq_row0, &seq_img,
                     &seq_branch, &lm_idx, &ptab, &kv, &calib_tok, &seg_pages, &win_end,
                     &score_logits, &score_idx, &score_k, &qz};
    for (DevBuf* b : all) free_buf(*b);
    if (pin) (void)hipHostFree(pin);
    for (auto& e : ev)
        if (e) (void)hipEventDestroy(e);
    for (auto& pr : prof_pending) {
        (void)hipEventDestroy(pr.second.first);
        (void)hipEventDestroy(pr.second.second);
    }
    for (hipEvent_t e : prof_free) (void)hipEventDestroy(e);
    for (auto& g : graphs)
        for (hipGraphExec_t e : g.exec)
            if (e) (void)hipGraphExecDestroy(e);
    if (ev_user) (void)hipEventDestroy(ev_user);
    if (ev_done) (void)hipEventDestroy(ev_done);
    if (stream) (void)hipStreamDestroy(stream);
}

namespace {

// ---------------------------------------------------------------- timing

hipEvent_t prof_event(hbsjd_ctx* c) {
    if (!c->prof_free.empty()) {
        hipEvent_t e = c->prof_free.back();
        c->prof_free.pop_back();
        return e;
    }
    hipEvent_t e = nullptr;
    (void)hipEventCreate(&e);
    return e;
}

// fold finished event pairs into the per-class totals
void prof_resolve(hbsjd_ctx* c) {
    if (c->prof_pending.empty()) return;
    (void)hipEventSynchronize(c->prof_pending.back().second.second);
    for (auto& pr : c->prof_pending) {
        float ms = 0.f;
        if (hipEventElapsedTime(&ms, pr.second.first, pr.second.second) == hipSuccess) {
            c->prof_ms[pr.first] += ms;
            c->prof_n[pr.first] += 1;
        }
        c->prof_free.push_back(pr.second.first);
        c->prof_free.push_back(pr.second.second);
    }
    c->prof_pending.clear();
}

// arms the launch-event slot for the one kernel launched inside this scope
// when its class is timed
struct Timed {
    hbsjd_ctx* c;
    int cls;
    bool armed = false;
    Timed(hbsjd_ctx* ctx, int k) : c(ctx), cls(k) {
        if ((c->prof_mask & (1u << k)) && c->prof_seen[k]++ % c->prof_every == 0) {
            LaunchEvents* ev = launch_events();
            ev->start = prof_event(c);
            ev->stop = prof_event(c);
            ev->used = false;
            armed = true;
        }
    }
    ~Timed() {
        if (!armed) return;
        LaunchEvents* ev = launch_events();
        if (ev->used) {
            c->prof_pending.push_back({cls, {ev->start, ev->stop}});
        } else {   // nothing was launched (empty row range)
            c->prof_free.push_back(ev->start);
            c->prof_free.push_back(ev->stop);
        }
        *ev = LaunchEvents{};
        if (c->prof_pending.size() >= 8192) prof_resolve(c);
    }
};

// ---------------------------------------------------------------- validation

std::string check_model(const hbsjd_model_desc& m) {
    if (m.n_layers < 1 || m.d_model < 4 || m.n_heads < 1 || m.mlp_hidden < 1 || m.vocab < 1 ||
        m.n_classes < 1 || m.grid < 1)
        return "model sizes must be positive";
    if (m.d_model % m.n_heads) return "d_model must be a multiple of n_heads";
    const int dh = m.d_model / m.n_heads;
    if (dh % 4) return "head_dim must be a multiple of 4";
    if (m.vocab > kMaxVocab) return "vocab must be <= 16384";
    if (m.vocab % 4) return "vocab must be a multiple of 4";
    if (m.dtype != HBSJD_DTYPE_F32 && m.dtype != HBSJD_DTYPE_BF16) return "unknown dtype";
    if (m.dtype == HBSJD_DTYPE_BF16) {
        if (dh != 64) return "a bf16 model needs head_dim 64";
        if (m.d_model % 64) return "a bf16 model needs d_model a multiple of 64";
        if (m.mlp_hidden % 64) return "a bf16 model needs mlp_hidden a multiple of 64";
        if (m.vocab % 64) return "a bf16 model needs vocab a multiple of 64";
    } else {
        if (dh > 64) return "fp32 needs head_dim <= 64";
        if ((long)m.grid * m.grid > 959) return "fp32 needs grid^2 <= 959";
    }
    if (!(m.rms_eps > 0.f) || !std::isfinite(m.rms_eps)) return "rms_eps must be positive";
    if (!(m.rope_base > 0.f) || !std::isfinite(m.rope_base)) return "rope_base must be positive";
    if ((long)m.grid * m.grid > 4096) return "grid too large";
    if (m.d_model > 1536) return "d_model must be <= 1536";
    return "";
}

size_t blob_floats(const hbsjd_ctx* c) {
    const size_t d = c->d, f = c->f, V = c->V, C = c->C, L = c->L;
    return V * d + (C + 1) * d + L * (2 * d + 3 * d * d + d * d + 3 * f * d) + d + V * d +
           (c->m.has_lm_bias ? V : 0);
}

// ---------------------------------------------------------------- forward

struct FwdRows {
    RowMeta meta;
    const int* nrows_dev;
    int nrows_cap;
    Segments seg;
    const int* nseg_dev;
    int nseg_cap;
    int max_rows_per_seg;
};

void* kv_layer(hbsjd_ctx* c, int l) {
    return (char*)c->kv.p + (size_t)l * c->kv_layer_elems * c->esz;
}

// decoder layers; leaves the residual stream in h and its final RMSNorm (gain
// g_out) in hb
void forward_layers(hbsjd_ctx* c, const FwdRows& r) {
    const bool bf = c->f16;
    hipStream_t s = c->stream;
    const int d = c->d, f = c->f;
    {
        Timed tm(c, HBSJD_K_EMBED);
        embed_norm(bf, r.meta, r.nrows_dev, r.nrows_cap, c->tok_emb, c->cls_emb, c->g_attn[0],
                   c->m.rms_eps, d, as<float>(c->h), c->hb.p, s);
    }
    const float* rc = as<float>(c->rope);
    const float* rs = rc + (size_t)(c->T + 1) * (c->dh / 2);
    for (int l = 0; l < c->L; ++l) {
        QkvArgs qa{c->qb.p, kv_layer(c, l), r.meta.pos, r.meta.kv, rc, rs, d, c->H, c->dh, c->T};
        {
            Timed tm(c, HBSJD_K_QKV);
            gemm_qkv(bf, c->hb.p, d, c->wqkv[l], c->s_qkv[l], 3 * d, d, r.nrows_dev, r.nrows_cap,
                     qa, s);
        }
        {
            Timed tm(c, HBSJD_K_ATTN);
            attention(bf, c->qb.p, c->ob.p, d, c->H, c->dh, kv_layer(c, l), as<int32_t>(c->ptab),
                      c->max_pages, r.seg, r.nseg_dev, r.nseg_cap, r.max_rows_per_seg, r.meta,
                      r.nrows_dev, r.nrows_cap, s);
        }
        // split-K applies to the MFMA path only; the fp32 path writes one partial
        const int so = bf ? split_for(r.nrows_cap, d, d) : 1;
        const int s2 = bf ? split_for(r.nrows_cap, d, f) : 1;
        {
            Timed tm(c, HBSJD_K_OPROJ);
            gemm_partial(bf, 0, c->ob.p, d, c->wo[l], c->s_o[l], d, d, r.nrows_dev, r.nrows_cap,
                         so, as<float>(c->part), s);
        }
        {
            Timed tm(c, HBSJD_K_NORM);
            reduce_residual_norm(bf, as<float>(c->part), so, r.nrows_cap, as<float>(c->h),
                                 r.nrows_dev, c->g_ffn[l], c->m.rms_eps, d, c->hb.p, s);
        }
        {
            Timed tm(c, HBSJD_K_W13);
            gemm_swiglu(bf, c->hb.p, d, c->w13[l], c->s_13[l], 2 * f, d, r.nrows_dev, r.nrows_cap,
                        c->act.p, s);
        }
        // With one K part the MFMA path adds W2 into the residual stream in its
        // epilogue and the norm only reads it (the same additions). O keeps
        // the partial sum: its launch is a single short round of tiles, whose
        // read-modify-write of the residual would sit exposed at its end
        // (XL: 42 + 24 us for O and its norm against 57 + 11).
        {
            Timed tm(c, HBSJD_K_W2);
            if (bf && s2 == 1)
                gemm_residual(1, c->act.p, f, c->w2[l], c->s_2[l], d, f, r.nrows_dev, r.nrows_cap,
                              as<float>(c->h), s);
            else
                gemm_partial(bf, 1, c->act.p, f, c->w2[l], c->s_2[l], d, f, r.nrows_dev,
                             r.nrows_cap, s2, as<float>(c->part), s);
        }
        {
            // the next layer's attention norm, or the final norm after the last layer
            Timed tm(c, HBSJD_K_NORM);
            reduce_residual_norm(bf, as<float>(c->part), bf && s2 == 1 ? 0 : s2, r.nrows_cap,
                                 as<float>(c->h), r.nrows_dev,
                                 l + 1 < c->L ? c->g_attn[l + 1] : c->g_out, c->m.rms_eps, d,
                                 c->hb.p, s);
        }
    }
}

// activation buffers for `rows` rows
hbsjd_status ensure_acts(hbsjd_ctx* c, long rows) {
    const size_t d = c->d, f = c->f;
    // kernels index activation rows with 32-bit element offsets
    if ((size_t)rows * std::max(3 * d, 2 * f) > (size_t)INT32_MAX)
        return fail(HBSJD_EINVAL, "too many rows in one forward for 32-bit element offsets");
    TRY(ensure(c, c->h, rows * d * 4));
    TRY(ensure(c, c->hb, rows * d * c->esz));
    TRY(ensure(c, c->qb, rows * d * c->esz));
    TRY(ensure(c, c->ob, rows * d * c->esz));
    TRY(ensure(c, c->act, rows * f * c->esz));
    TRY(ensure(c, c->row_tok, rows * 4));
    TRY(ensure(c, c->row_pos, rows * 4));
    TRY(ensure(c, c->row_kv, rows * 4));
    TRY(ensure(c, c->row_seq, rows * 4));
    const long sp = c->f16 ? std::max(split_for((int)rows, c->d, c->d),
                                       split_for((int)rows, c->d, c->f))
                            : 1;
    TRY(ensure(c, c->part, (size_t)sp * rows * d * 4));
    return HBSJD_OK;
}

// page table and KV pool for n_seq sequences of cap positions each
hbsjd_status ensure_kv(hbsjd_ctx* c, int n_seq, int cap) {
    c->max_pages = (cap + kPage - 1) / kPage;
    const long pages = (long)n_seq * c->max_pages;
    const long page_elems = 2L * kPage * c->d;
    c->kv_layer_elems = pages * page_elems;
    // kernels address a layer's pool with 32-bit element offsets
    if (c->kv_layer_elems > (long)INT32_MAX)
        return fail(HBSJD_EINVAL, "KV pool of one layer above 2^31 elements");
    const size_t bytes = (size_t)c->L * c->kv_layer_elems * c->esz;
    if (c->max_kv_bytes && bytes > c->max_kv_bytes)
        return fail(HBSJD_ENOMEM, "KV cache needs " + std::to_string(bytes) +
                                      " bytes, above the context's cap");
    const bool grow = c->kv.n < bytes;
    TRY(ensure(c, c->kv, bytes));
    if (grow) HIPTRY(c, hipMemsetAsync(c->kv.p, 0, c->kv.n, c->stream));
    // page of (sequence q, tile j) = j * n_seq + q: pages of one sequence are not adjacent
    std::vector<int32_t> pt((size_t)n_seq * c->max_pages);
    for (int q = 0; q < n_seq; ++q)
        for (int j = 0; j < c->max_pages; ++j) pt[(size_t)q * c->max_pages + j] = j * n_seq + q;
    TRY(ensure(c, c->ptab, pt.size() * 4));
    HIPTRY(c, hipMemcpyAsync(c->ptab.p, pt.data(), pt.size() * 4, hipMemcpyHostToDevice, c->stream));
    HIPTRY(c, hipStreamSynchronize(c->stream));
    return HBSJD_OK;
}

hbsjd_status check_device_error(hbsjd_ctx* c) {
    int32_t err = 0;
    HIPTRY(c, hipMemcpyAsync(&err, as<int32_t>(c->meta) + kMetaError, 4, hipMemcpyDeviceToHost,
                             c->stream));
    HIPTRY(c, hipStreamSynchronize(c->stream));
    if (err) {
        c->poisoned = true;
        std::string why;
        if (err & kErrNanLogit) why += " NaN logit;";
        if (err & kErrZeroProposal) why += " zero proposal probability of a reused draft;";
        if (err & kErrBadToken) why += " token out of range;";
        if (err & kErrRoundOverflow) why += " more rounds than max_rounds;";
        return fail(HBSJD_EINTERNAL, "device check failed:" + why);
    }
    return HBSJD_OK;
}

// ---------------------------------------------------------------- rollout set-up

hbsjd_status validate_args(const hbsjd_ctx* c, const hbsjd_rollout_args* a) {
    if (!a) return fail(HBSJD_EINVAL, "args is NULL");
    if (a->batch < 1) return fail(HBSJD_EINVAL, "batch must be >= 1");
    if (a->verify_mode < HBSJD_VERIFY_PROB || a->verify_mode > HBSJD_VERIFY_AR_GREEDY)
        return fail(HBSJD_EINVAL, "unknown verify_mode");
    const bool ar = a->verify_mode >= HBSJD_VERIFY_AR;
    if (!ar && (a->window < 1 || a->window > 64)) return fail(HBSJD_EINVAL, "window must be in [1, 64]");
    if (!ar && a->history < 1) return fail(HBSJD_EINVAL, "history must be >= 1");
    if (a->top_k < 0) return fail(HBSJD_EINVAL, "top_k must be >= 0");
    if (!std::isfinite(a->cfg_scale)) return fail(HBSJD_EINVAL, "cfg_scale must be finite");
    if (a->exec_mode < HBSJD_EXEC_AUTO || a->exec_mode > HBSJD_EXEC_COMPACT)
        return fail(HBSJD_EINVAL, "unknown exec_mode");
    if (a->gamma < -1) return fail(HBSJD_EINVAL, "gamma must be >= -1");
    if (a->progress != HBSJD_PROGRESS_INDEPENDENT && a->progress != HBSJD_PROGRESS_SYNC)
        return fail(HBSJD_EINVAL, "unknown progress mode");
    if (!a->prefix_tokens || !a->prefix_len || !a->class_labels || !a->temperature)
        return fail(HBSJD_EINVAL, "prefix_tokens, prefix_len, class_labels and temperature are required");
    if (!c->f16 && c->T + (ar ? 0 : a->window) + 1 > 1024)
        return fail(HBSJD_EINVAL, "fp32 mode supports T + window + 1 <= 1024");
    int need = 0;
    for (int b = 0; b < a->batch; ++b) {
        const int k = a->prefix_len[b];
        if (k < 0 || k > c->T) return fail(HBSJD_EINVAL, "prefix_len out of [0, T]");
        if (a->class_labels[b] < 0 || a->class_labels[b] >= c->C)
            return fail(HBSJD_EINVAL, "class label out of [0, n_classes)");
        const float tau = a->temperature[b];
        if (!std::isfinite(tau) || !(tau > 0.f))
            return fail(HBSJD_EINVAL, "temperature must be finite and > 0");
        need = std::max(need, c->T - k);
    }
    if (a->max_rounds < need) return fail(HBSJD_EINVAL, "max_rounds below max_b (T - k_b)");
    return HBSJD_OK;
}

// The products of the calling thread take a row bound until the end of
// scope: an upper bound of a round's rows, or the exact rows of a forward whose
// row count the host set itself.
struct RowBound {
    explicit RowBound(int rows) { gemm_row_bound(rows); }
    ~RowBound() { gemm_row_bound(-1); }
};

hbsjd_status begin(hbsjd_ctx* c, const hbsjd_rollout_args* a, int32_t* counts_dev) {
    if (!c->weights) return fail(HBSJD_ESTATE, "weights not loaded");
    TRY(validate_args(c, a));
    hipStream_t s = c->stream;
    const bool ar = a->verify_mode >= HBSJD_VERIFY_AR;
    const int B = a->batch, T = c->T, W = ar ? 0 : a->window;
    c->have_state = false;
    c->B = B;
    c->W = W;
    c->ar = ar;
    c->sync = !ar && a->progress == HBSJD_PROGRESS_SYNC;
    c->Hh = ar ? 1 : a->history;
    c->top_k = a->top_k;
    c->cfg = a->cfg_scale != 0.f ? 2 : 1;
    c->cfg_scale = a->cfg_scale;
    c->greedy = a->verify_mode == HBSJD_VERIFY_GREEDY || a->verify_mode == HBSJD_VERIFY_AR_GREEDY;
    c->exec_mode = a->exec_mode;
    c->gamma = a->gamma >= 0 ? a->gamma : (c->gamma_cal >= 0 ? c->gamma_cal : B / 2);
    c->seed = a->seed;
    HIPTRY(c, hipEventRecord(c->ev_user, c->user_stream));
    HIPTRY(c, hipStreamWaitEvent(c->stream, c->ev_user, 0));
    c->max_rounds = a->max_rounds;
    c->rounds_launched = 0;
    c->a_bound = B;
    const int cfg = c->cfg;
    const int S = B * cfg;

    // prefill geometry (host knows the lengths)
    std::vector<int32_t> row0(1, 0), simg, sbr, lidx, pslots;
    int maxlen = 0;
    // SJD prefills positions 0..k_b and drafts from the logits at k_b; the AR
    // baseline prefills 0..k_b-1 and its first round forwards position k_b
    for (int b = 0; b < B; ++b) {
        const int k = a->prefix_len[b];
        const int pre = ar ? k : k + 1;
        if (k >= T || pre == 0) continue;
        pslots.push_back(b);
        for (int br = 0; br < cfg; ++br) {
            simg.push_back(b);
            sbr.push_back(br);
            lidx.push_back(row0.back() + pre - 1);
            row0.push_back(row0.back() + pre);
        }
        maxlen = std::max(maxlen, pre);
    }
    const int n_seq = (int)simg.size();
    const int pf_rows = row0.back();
    const long round_rows = (long)S * (W + 1);
    const long out_rows = (long)B * (W + 1);

    TRY(ensure_acts(c, std::max<long>(pf_rows, round_rows)));
    TRY(ensure_kv(c, S, T + W + 1));
    TRY(ensure(c, c->seg_pages, (size_t)std::max(S, n_seq) * c->max_pages * 4));
    TRY(ensure(c, c->xtok, (size_t)B * T * 4));
    TRY(ensure(c, c->cursor, B * 4));
    TRY(ensure(c, c->drafts, (size_t)B * W * 4));
    TRY(ensure(c, c->qsrc, (size_t)B * W * 4));
    TRY(ensure(c, c->labels, B * 4));
    TRY(ensure(c, c->temps, B * 4));
    TRY(ensure(c, c->plen, B * 4));
    if (c->sync) TRY(ensure(c, c->win_end, B * 4));
    TRY(ensure(c, c->meta, kMetaCount * 4));
    TRY(ensure(c, c->meta_pf, kMetaCount * 4));
    TRY(ensure(c, c->a_hist, (size_t)(a->max_rounds + 1) * 4));
    TRY(ensure(c, c->mode_hist, (size_t)(a->max_rounds + 1) * 4));
    TRY(ensure(c, c->stats, 4 * 8));
    TRY(ensure(c, c->seg_seq, S * 4));
    TRY(ensure(c, c->seg_row0, std::max(S, n_seq + 1) * 4));
    TRY(ensure(c, c->seg_nrows, S * 4));
    TRY(ensure(c, c->seg_pos0, S * 4));
    TRY(ensure(c, c->slot_img, B * 4));
    TRY(ensure(c, c->active_list, B * 4));
    TRY(ensure(c, c->pf_slots, B * 4));
    TRY(ensure(c, c->seq_row0, (n_seq + 1) * 4));
    TRY(ensure(c, c->seq_img, std::max(n_seq, 1) * 4));
    TRY(ensure(c, c->seq_branch, std::max(n_seq, 1) * 4));
    TRY(ensure(c, c->lm_idx, std::max(n_seq, 1) * 4));
    for (int k = 0; k < 2; ++k) {
        TRY(ensure(c, c->P[k], (size_t)(cfg == 1 ? round_rows : out_rows) * c->V * 4));
        TRY(ensure(c, c->amax[k], (size_t)out_rows * 4));
    }
    TRY(ensure(c, c->samp, (size_t)out_rows * 4));
    if (cfg == 2) TRY(ensure(c, c->logits, (size_t)round_rows * c->V * 4));
    (void)counts_dev;
    TRY(ensure(c, c->counts_own, (size_t)a->max_rounds * B * 4));
    c->counts = as<int32_t>(c->counts_own);
    if (!c->pin) {
        HIPTRY(c, hipHostMalloc((void**)&c->pin, 64, hipHostMallocDefault));
        HIPTRY(c, hipEventCreateWithFlags(&c->ev[0], hipEventDisableTiming));
        HIPTRY(c, hipEventCreateWithFlags(&c->ev[1], hipEventDisableTiming));
    }

    // state
    std::vector<int32_t> meta(kMetaCount, 0);
    meta[kMetaRound] = -1;
    meta[kMetaGamma] = c->gamma;
    meta[kMetaExec] = c->exec_mode;
    meta[kMetaSeedLo] = (int32_t)(uint32_t)c->seed;
    meta[kMetaSeedHi] = (int32_t)(uint32_t)(c->seed >> 32);
    HIPTRY(c, hipMemcpyAsync(c->meta.p, meta.data(), kMetaCount * 4, hipMemcpyHostToDevice, s));
    HIPTRY(c, hipMemcpyAsync(c->xtok.p, a->prefix_tokens, (size_t)B * T * 4, hipMemcpyDeviceToDevice, s));
    HIPTRY(c, hipMemcpyAsync(c->cursor.p, a->prefix_len, B * 4, hipMemcpyHostToDevice, s));
    HIPTRY(c, hipMemcpyAsync(c->plen.p, a->prefix_len, B * 4, hipMemcpyHostToDevice, s));
    std::vector<int32_t> wend;   // first window of each image: positions k_b+1 .. min(k_b+W, T)
    if (c->sync) {
        wend.resize(B);
        for (int b = 0; b < B; ++b) wend[b] = std::min(a->prefix_len[b] + W, T);
        HIPTRY(c, hipMemcpyAsync(c->win_end.p, wend.data(), B * 4, hipMemcpyHostToDevice, s));
    }
    HIPTRY(c, hipMemcpyAsync(c->labels.p, a->class_labels, B * 4, hipMemcpyHostToDevice, s));
    HIPTRY(c, hipMemcpyAsync(c->temps.p, a->temperature, B * 4, hipMemcpyHostToDevice, s));
    HIPTRY(c, hipMemsetAsync(c->drafts.p, 0xff, (size_t)B * W * 4, s));
    HIPTRY(c, hipMemsetAsync(c->qsrc.p, 0xff, (size_t)B * W * 4, s));
    HIPTRY(c, hipMemsetAsync(c->stats.p, 0, 32, s));
    HIPTRY(c, hipMemsetAsync(c->counts, 0, (size_t)a->max_rounds * B * 4, s));
    check_prefix(as<int32_t>(c->xtok), as<int32_t>(c->plen), B, T, c->V,
                 as<int32_t>(c->meta) + kMetaError, s);
    {
        int32_t err = 0;
        HIPTRY(c, hipMemcpyAsync(&err, as<int32_t>(c->meta) + kMetaError, 4, hipMemcpyDeviceToHost, s));
        HIPTRY(c, hipStreamSynchronize(s));
        if (err) return fail(HBSJD_EINVAL, "a prefix token is outside [0, vocab)");
    }
    if (n_seq == 0) {
        c->have_state = true;
        return HBSJD_OK;
    }

    // prefill rows and segments
    std::vector<int32_t> segseq(n_seq), segrow0(n_seq), segn(n_seq), segpos(n_seq, 0);
    for (int q = 0; q < n_seq; ++q) {
        segseq[q] = simg[q] * cfg + sbr[q];
        segrow0[q] = row0[q];
        segn[q] = row0[q + 1] - row0[q];
    }
    HIPTRY(c, hipMemcpyAsync(c->seq_row0.p, row0.data(), (n_seq + 1) * 4, hipMemcpyHostToDevice, s));
    HIPTRY(c, hipMemcpyAsync(c->seq_img.p, simg.data(), n_seq * 4, hipMemcpyHostToDevice, s));
    HIPTRY(c, hipMemcpyAsync(c->seq_branch.p, sbr.data(), n_seq * 4, hipMemcpyHostToDevice, s));
    HIPTRY(c, hipMemcpyAsync(c->lm_idx.p, lidx.data(), n_seq * 4, hipMemcpyHostToDevice, s));
    HIPTRY(c, hipMemcpyAsync(c->pf_slots.p, pslots.data(), pslots.size() * 4, hipMemcpyHostToDevice, s));
    HIPTRY(c, hipMemcpyAsync(c->seg_seq.p, segseq.data(), n_seq * 4, hipMemcpyHostToDevice, s));
    HIPTRY(c, hipMemcpyAsync(c->seg_row0.p, segrow0.data(), n_seq * 4, hipMemcpyHostToDevice, s));
    HIPTRY(c, hipMemcpyAsync(c->seg_nrows.p, segn.data(), n_seq * 4, hipMemcpyHostToDevice, s));
    HIPTRY(c, hipMemcpyAsync(c->seg_pos0.p, segpos.data(), n_seq * 4, hipMemcpyHostToDevice, s));
    seg_pages(as<int32_t>(c->seg_seq), n_seq, as<int32_t>(c->ptab), c->max_pages,
              as<int32_t>(c->seg_pages), s);
    std::vector<int32_t> mpf(kMetaCount, 0);
    mpf[kMetaRows] = pf_rows;
    mpf[kMetaSegs] = n_seq;
    mpf[kMetaOutRows] = (int)pslots.size();
    mpf[kMetaImgs] = (int)pslots.size();
    mpf[kMetaActive] = n_seq;     // rows of the lm_head
    HIPTRY(c, hipMemcpyAsync(c->meta_pf.p, mpf.data(), kMetaCount * 4, hipMemcpyHostToDevice, s));
    // the host staging vectors must outlive the async copies
    HIPTRY(c, hipStreamSynchronize(s));

    PrefillRowsArgs pa{n_seq, T, cfg, c->C, c->max_pages, pf_rows, as<int32_t>(c->seq_row0),
                       as<int32_t>(c->seq_img), as<int32_t>(c->seq_branch), as<int32_t>(c->xtok),
                       as<int32_t>(c->labels), as<int32_t>(c->ptab), as<int32_t>(c->row_tok),
                       as<int32_t>(c->row_pos), as<int32_t>(c->row_kv), as<int32_t>(c->row_seq)};
    prefill_rows(pa, s);
    int32_t* mp = as<int32_t>(c->meta_pf);
    FwdRows fr{RowMeta{as<int32_t>(c->row_tok), as<int32_t>(c->row_pos), as<int32_t>(c->row_kv),
                       as<int32_t>(c->row_seq)},
               mp + kMetaRows, pf_rows,
               Segments{as<int32_t>(c->seg_seq), as<int32_t>(c->seg_row0), as<int32_t>(c->seg_nrows),
                        as<int32_t>(c->seg_pos0), as<int32_t>(c->seg_pages)},
               mp + kMetaSegs, n_seq, maxlen};
    RowBound rb(pf_rows);
    forward_layers(c, fr);
    if (ar) {   // the prefill only fills the cache
        HIPTRY(c, hipGetLastError());
        c->have_state = true;
        return HBSJD_OK;
    }
    // final norm of each sequence's last row, lm_head, transform, first window
    rmsnorm(c->f16, as<float>(c->h), as<int32_t>(c->lm_idx), mp + kMetaActive, n_seq, c->g_out,
            c->m.rms_eps, c->d, c->hb.p, s);
    float* lg = cfg == 1 ? as<float>(c->P[1]) : as<float>(c->logits);
    gemm_logits(c->f16, c->hb.p, c->d, c->w_lm, c->s_lm, c->V, c->d, mp + kMetaActive, n_seq, lg, c->b_lm, s);
    TransformArgs ta{lg, as<float>(c->P[1]), as<int32_t>(c->amax[1]),
                     as<int32_t>(c->samp), as<int32_t>(c->pf_slots), as<int32_t>(c->cursor),
                     as<float>(c->temps), 1, cfg, c->V, c->top_k, T, c->cfg_scale,
                     mp + kMetaOutRows, (int)pslots.size(), as<int32_t>(c->meta)};
    transform(ta, s);
    VerifyArgs va{B, W, T, c->Hh, c->V, c->greedy, 1, 1, c->max_rounds,
                  as<float>(c->P[1]), as<int32_t>(c->amax[1]),
                  as<int32_t>(c->samp), nullptr, as<int32_t>(c->pf_slots), mp + kMetaImgs,
                  (int)pslots.size(),
                  as<int32_t>(c->cursor), as<int32_t>(c->xtok), as<int32_t>(c->drafts),
                  as<int32_t>(c->qsrc), nullptr, as<int64_t>(c->stats), as<int32_t>(c->meta)};
    verify_commit(va, s);
    HIPTRY(c, hipGetLastError());
    c->have_state = true;
    return HBSJD_OK;
}

// An upper bound of the next round's rows: every slot when the round can run
// Full, else the rows of at most a_bound active images.
int round_row_bound(const hbsjd_ctx* c) {
    const bool full = c->exec_mode == HBSJD_EXEC_FULL ||
                      (c->exec_mode == HBSJD_EXEC_AUTO && c->a_bound > c->gamma);
    return (full ? c->B : std::min(c->a_bound, c->B)) * c->cfg * (c->W + 1);
}


// queue the launches of one round on buffer parity `cur`; every launch sizes
// itself from the device counts the round's set-up kernel writes
void enqueue_round(hbsjd_ctx* c, int cur, bool with_verify = true) {
    hipStream_t s = c->stream;
    RowBound rb(round_row_bound(c));
    const int B = c->B, W = c->W, cfg = c->cfg, S = B * cfg, R = W + 1;
    int32_t* mt = as<int32_t>(c->meta);
    RoundSetupArgs sa{B, W, c->T, cfg, c->C, c->max_pages, c->max_rounds,
                      as<int32_t>(c->cursor), as<int32_t>(c->drafts), as<int32_t>(c->xtok),
                      as<int32_t>(c->labels), as<int32_t>(c->ptab), as<int32_t>(c->slot_img),
                      as<int32_t>(c->active_list), as<int32_t>(c->row_tok), as<int32_t>(c->row_pos),
                      as<int32_t>(c->row_kv), as<int32_t>(c->row_seq), as<int32_t>(c->seg_seq),
                      as<int32_t>(c->seg_row0), as<int32_t>(c->seg_nrows), as<int32_t>(c->seg_pos0),
                      mt, as<int32_t>(c->a_hist), as<int32_t>(c->mode_hist),
                      as<int32_t>(c->seg_pages), c->sync ? as<int32_t>(c->win_end) : nullptr};
    {
        Timed tm(c, HBSJD_K_SETUP);
        round_setup(sa, s);
    }
    const int rows_cap = S * R;
    FwdRows fr{RowMeta{as<int32_t>(c->row_tok), as<int32_t>(c->row_pos), as<int32_t>(c->row_kv),
                       as<int32_t>(c->row_seq)},
               mt + kMetaRows, rows_cap,
               Segments{as<int32_t>(c->seg_seq), as<int32_t>(c->seg_row0), as<int32_t>(c->seg_nrows),
                        as<int32_t>(c->seg_pos0), as<int32_t>(c->seg_pages)},
               mt + kMetaSegs, S, R};
    forward_layers(c, fr);
    float* lg = cfg == 1 ? as<float>(c->P[cur]) : as<float>(c->logits);
    {
        Timed tm(c, HBSJD_K_LMHEAD);
        gemm_logits(c->f16, c->hb.p, c->d, c->w_lm, c->s_lm, c->V, c->d, mt + kMetaRows, rows_cap, lg,
                    c->b_lm, s);
    }
    TransformArgs ta{lg, as<float>(c->P[cur]), as<int32_t>(c->amax[cur]),
                     as<int32_t>(c->samp), as<int32_t>(c->slot_img), as<int32_t>(c->cursor),
                     as<float>(c->temps), R, cfg, c->V, c->top_k, c->T, c->cfg_scale,
                     mt + kMetaOutRows, B * R, mt};
    {
        Timed tm(c, HBSJD_K_TRANSFORM);
        transform(ta, s);
    }
    if (!with_verify) return;
    VerifyArgs va{B, W, c->T, c->Hh, c->V, c->greedy, 0, R, c->max_rounds,
                  as<float>(c->P[cur]), as<int32_t>(c->amax[cur]),
                  as<int32_t>(c->samp), as<float>(c->P[cur ^ 1]), as<int32_t>(c->slot_img),
                  mt + kMetaImgs, B,
                  as<int32_t>(c->cursor), as<int32_t>(c->xtok), as<int32_t>(c->drafts),
                  as<int32_t>(c->qsrc), c->counts, as<int64_t>(c->stats), mt, c->ar,
                  c->sync ? as<int32_t>(c->win_end) : nullptr};
    {
        Timed tm(c, HBSJD_K_VERIFY);
        verify_commit(va, s);
    }
}

// everything a captured round bakes into its kernel arguments
std::vector<uint64_t> graph_signature(hbsjd_ctx* c) {
    std::vector<uint64_t> g = {(uint64_t)c->B, (uint64_t)c->W, (uint64_t)c->cfg,
                               (uint64_t)c->Hh, (uint64_t)c->top_k, (uint64_t)c->greedy,
                               (uint64_t)c->ar, (uint64_t)c->sync,
                               (uint64_t)c->max_rounds, (uint64_t)c->max_pages,
                               (uint64_t)c->kv_layer_elems};
    uint32_t cs;
    std::memcpy(&cs, &c->cfg_scale, 4);
    g.push_back(cs);
    DevBuf* bufs[] = {&c->xtok, &c->cursor, &c->drafts, &c->qsrc, &c->labels, &c->temps,
                      &c->meta, &c->a_hist, &c->mode_hist, &c->stats, &c->counts_own,
                      &c->row_tok, &c->row_pos, &c->row_kv, &c->row_seq, &c->seg_seq,
                      &c->seg_row0, &c->seg_nrows, &c->seg_pos0, &c->slot_img,
                      &c->active_list, &c->h, &c->hb, &c->qb, &c->ob, &c->act, &c->part,
                      &c->P[0], &c->P[1], &c->amax[0], &c->amax[1],
                      &c->samp, &c->logits, &c->ptab, &c->kv, &c->wbuf, &c->rope, &c->win_end,
                      &c->seg_pages};
    for (DevBuf* b : bufs) g.push_back((uint64_t)(uintptr_t)b->p);
    return g;
}

void drop_round_graphs(hbsjd_ctx* c) {
    for (auto& g : c->graphs)
        for (hipGraphExec_t e : g.exec)
            if (e) (void)hipGraphExecDestroy(e);
    c->graphs.clear();
    c->gsig.clear();
}

// the products' kernels for a row bound match those a pair was captured with
bool plan_holds(const std::vector<GemmPlan>& plan, int row_bound) {
    for (const GemmPlan& p : plan)
        if (gemm_plan(p, row_bound) != p.kernels) return false;
    return true;
}

// while alive, the calling thread's products record their kernels in `log`
struct PlanLog {
    explicit PlanLog(std::vector<GemmPlan>* log) { gemm_plan_log(log); }
    ~PlanLog() { gemm_plan_log(nullptr); }
};

// capture the round, under the current row bound, as one more pair of graphs
// (the pairs of other bounds are kept, up to kMaxRoundGraphs)
constexpr size_t kMaxRoundGraphs = 8;
hbsjd_status capture_round_graphs(hbsjd_ctx* c) {
    if (c->graphs.size() >= kMaxRoundGraphs) drop_round_graphs(c);
    hbsjd_ctx::RoundGraphs g;
    for (int par = 0; par < 2; ++par) {
        hipGraph_t graph = nullptr;
        std::vector<GemmPlan> log;
        hipError_t e = hipStreamBeginCapture(c->stream, hipStreamCaptureModeThreadLocal);
        if (e == hipSuccess) {
            PlanLog pl(&log);
            enqueue_round(c, par);
            e = hipStreamEndCapture(c->stream, &graph);
        }
        if (e == hipSuccess) {
            e = hipGraphInstantiate(&g.exec[par], graph, nullptr, nullptr, 0);
            (void)hipGraphDestroy(graph);
        }
        if (e != hipSuccess) {
            for (hipGraphExec_t x : g.exec)
                if (x) (void)hipGraphExecDestroy(x);
            return hip_fail(c, e, "round graph capture");
        }
        if (par == 0) g.plan = std::move(log);
    }
    g.bound = round_row_bound(c);
    c->graphs.push_back(std::move(g));
    return HBSJD_OK;
}

// queue one round: a graph replay, or eager launches while kernels are timed
hbsjd_status launch_round(hbsjd_ctx* c) {
    const int cur = c->rounds_launched & 1;
    if (c->use_graphs && c->prof_mask == 0) {
        std::vector<uint64_t> sig = graph_signature(c);
        if (c->gsig != sig) {
            drop_round_graphs(c);
            c->gsig = std::move(sig);
        }
        const int bound = round_row_bound(c);
        hbsjd_ctx::RoundGraphs* g = nullptr;
        for (auto& x : c->graphs)
            if (x.bound >= bound && plan_holds(x.plan, bound)) {
                g = &x;
                break;
            }
        if (!g) {
            TRY(capture_round_graphs(c));
            g = &c->graphs.back();
        }
        HIPTRY(c, hipGraphLaunch(g->exec[cur], c->stream));
    } else {
        enqueue_round(c, cur);
        HIPTRY(c, hipGetLastError());
    }
    c->rounds_launched += 1;
    return HBSJD_OK;
}

// Teacher-forced forward through every layer. Sequence q is image simg[q]:
// [class labels[image], tokens[image][0 .. lens[q]-1]] at positions 0..lens[q],
// rows row0[q] .. row0[q+1]-1; its KV pages are those of sequence `image`.
// check_len[image] prefix tokens of each image are range-checked first. Leaves
// the final residual stream in c->h, its normed rows in c->hb and the row
// count in meta_pf. Synchronous up to the layers' launches.
hbsjd_status forward_core(hbsjd_ctx* c, int n_images, const int32_t* tokens,
                          const std::vector<int32_t>& labels, const std::vector<int32_t>& check_len,
                          const std::vector<int32_t>& simg, const std::vector<int32_t>& lens,
                          std::vector<int32_t>& row0) {
    const int n_seqs = (int)simg.size();
    row0.assign(1, 0);
    int maxlen = 0;
    for (int q = 0; q < n_seqs; ++q) {
        row0.push_back(row0.back() + lens[q] + 1);
        maxlen = std::max(maxlen, lens[q] + 1);
    }
    hipStream_t s = c->stream;
    const int rows = row0.back();
    c->have_state = false;
    HIPTRY(c, hipEventRecord(c->ev_user, c->user_stream));
    HIPTRY(c, hipStreamWaitEvent(c->stream, c->ev_user, 0));
    TRY(ensure_acts(c, rows));
    TRY(ensure_kv(c, n_images, c->T + 1));
    TRY(ensure(c, c->meta, kMetaCount * 4));
    TRY(ensure(c, c->meta_pf, kMetaCount * 4));
    TRY(ensure(c, c->plen, n_images * 4));
    TRY(ensure(c, c->labels, n_images * 4));
    TRY(ensure(c, c->seq_row0, (n_seqs + 1) * 4));
    TRY(ensure(c, c->seq_img, n_seqs * 4));
    TRY(ensure(c, c->seq_branch, n_seqs * 4));
    TRY(ensure(c, c->seg_seq, n_seqs * 4));
    TRY(ensure(c, c->seg_row0, (n_seqs + 1) * 4));
    TRY(ensure(c, c->seg_nrows, n_seqs * 4));
    TRY(ensure(c, c->seg_pos0, n_seqs * 4));
    TRY(ensure(c, c->seg_pages, (size_t)n_seqs * c->max_pages * 4));
    std::vector<int32_t> segn(n_seqs), segpos(n_seqs, 0), sbr(n_seqs, 0), mz(kMetaCount, 0);
    for (int q = 0; q < n_seqs; ++q) segn[q] = row0[q + 1] - row0[q];
    HIPTRY(c, hipMemcpyAsync(c->meta.p, mz.data(), kMetaCount * 4, hipMemcpyHostToDevice, s));
    HIPTRY(c, hipMemcpyAsync(c->plen.p, check_len.data(), n_images * 4, hipMemcpyHostToDevice, s));
    check_prefix(tokens, as<int32_t>(c->plen), n_images, c->T, c->V, as<int32_t>(c->meta) + kMetaError, s);
    int32_t err = 0;
    HIPTRY(c, hipMemcpyAsync(&err, as<int32_t>(c->meta) + kMetaError, 4, hipMemcpyDeviceToHost, s));
    HIPTRY(c, hipStreamSynchronize(s));
    if (err) return fail(HBSJD_EINVAL, "a token is outside [0, vocab)");
    HIPTRY(c, hipMemcpyAsync(c->labels.p, labels.data(), n_images * 4, hipMemcpyHostToDevice, s));
    HIPTRY(c, hipMemcpyAsync(c->seq_row0.p, row0.data(), (n_seqs + 1) * 4, hipMemcpyHostToDevice, s));
    HIPTRY(c, hipMemcpyAsync(c->seq_img.p, simg.data(), n_seqs * 4, hipMemcpyHostToDevice, s));
    HIPTRY(c, hipMemcpyAsync(c->seq_branch.p, sbr.data(), n_seqs * 4, hipMemcpyHostToDevice, s));
    HIPTRY(c, hipMemcpyAsync(c->seg_seq.p, simg.data(), n_seqs * 4, hipMemcpyHostToDevice, s));
    HIPTRY(c, hipMemcpyAsync(c->seg_row0.p, row0.data(), n_seqs * 4, hipMemcpyHostToDevice, s));
    HIPTRY(c, hipMemcpyAsync(c->seg_nrows.p, segn.data(), n_seqs * 4, hipMemcpyHostToDevice, s));
    HIPTRY(c, hipMemcpyAsync(c->seg_pos0.p, segpos.data(), n_seqs * 4, hipMemcpyHostToDevice, s));
    seg_pages(as<int32_t>(c->seg_seq), n_seqs, as<int32_t>(c->ptab), c->max_pages,
              as<int32_t>(c->seg_pages), s);
    std::vector<int32_t> mpf(kMetaCount, 0);
    mpf[kMetaRows] = rows;
    mpf[kMetaSegs] = n_seqs;
    HIPTRY(c, hipMemcpyAsync(c->meta_pf.p, mpf.data(), kMetaCount * 4, hipMemcpyHostToDevice, s));
    HIPTRY(c, hipStreamSynchronize(s));
    // C is the null class here; the row builder maps branch 0 to labels[image]
    PrefillRowsArgs pa{n_seqs, c->T, 1, c->C, c->max_pages, rows, as<int32_t>(c->seq_row0),
                       as<int32_t>(c->seq_img), as<int32_t>(c->seq_branch), tokens,
                       as<int32_t>(c->labels), as<int32_t>(c->ptab), as<int32_t>(c->row_tok),
                       as<int32_t>(c->row_pos), as<int32_t>(c->row_kv), as<int32_t>(c->row_seq)};
    prefill_rows(pa, s);
    int32_t* mp = as<int32_t>(c->meta_pf);
    FwdRows fr{RowMeta{as<int32_t>(c->row_tok), as<int32_t>(c->row_pos), as<int32_t>(c->row_kv),
                       as<int32_t>(c->row_seq)},
               mp + kMetaRows, rows,
               Segments{as<int32_t>(c->seg_seq), as<int32_t>(c->seg_row0),
                        as<int32_t>(c->seg_nrows), as<int32_t>(c->seg_pos0), as<int32_t>(c->seg_pages)},
               mp + kMetaSegs, n_seqs, maxlen};
    RowBound rb(rows);
    forward_layers(c, fr);
    HIPTRY(c, hipGetLastError());
    return HBSJD_OK;
}

#define GUARD(ctx)                                                                       \
    if (!(ctx)) return fail(HBSJD_EINVAL, "ctx is NULL");                                \
    if ((ctx)->poisoned) return fail(HBSJD_ESTATE, "context is poisoned by an earlier failure"); \
    HIPTRY(ctx, hipSetDevice((ctx)->device))

}  // namespace

// ==================================================================== C ABI

extern "C" {

const char* hbsjd_last_error(void) { return g_err.c_str(); }

const char* hbsjd_version(void) { return "hbsjd-gfx950 0.1"; }

hbsjd_status hbsjd_create(const hbsjd_model_desc* m, uint64_t max_kv_bytes, void* stream,
                          hbsjd_ctx** out) {
    try {
        if (!m || !out) return fail(HBSJD_EINVAL, "model and out must not be NULL");
        *out = nullptr;
        const std::string why = check_model(*m);
        if (!why.empty()) return fail(HBSJD_EINVAL, why);
        hbsjd_ctx* c = new hbsjd_ctx();
        c->m = *m;
        c->L = m->n_layers;
        c->d = m->d_model;
        c->H = m->n_heads;
        c->dh = m->d_model / m->n_heads;
        c->f = m->mlp_hidden;
        c->V = m->vocab;
        c->C = m->n_classes;
        c->G = m->grid;
        c->T = m->grid * m->grid;
        c->nC = (c->V + kChunk - 1) / kChunk;
        c->f16 = m->dtype == HBSJD_DTYPE_BF16;
        c->esz = c->f16 ? 2 : 4;
        c->user_stream = (hipStream_t)stream;
        c->max_kv_bytes = max_kv_bytes;
        hipError_t e = hipGetDevice(&c->device);
        if (e == hipSuccess) e = gemm_setup();
        attention_setup();
        if (e == hipSuccess) e = hipStreamCreateWithFlags(&c->stream, hipStreamNonBlocking);
        if (e == hipSuccess) e = hipEventCreateWithFlags(&c->ev_user, hipEventDisableTiming);
        if (e != hipSuccess) {
            delete c;
            return fail(HBSJD_EHIP, std::string("stream set-up: ") + hipGetErrorString(e));
        }
        if (const char* g = std::getenv("HBSJD_NO_GRAPHS")) c->use_graphs = !(g[0] == '1');
        // 2D RoPE tables: position s >= 1 is grid cell (row, col) = divmod(s - 1, G);
        // pair i < dh/4 turns by row * base^(-4i/dh), pair i >= dh/4 by
        // col * base^(-4(i - dh/4)/dh); position 0 (class token) is not turned.
        const int half = c->dh / 2, quarter = c->dh / 4;
        std::vector<float> tab((size_t)2 * (c->T + 1) * half);
        float* cs = tab.data();
        float* sn = tab.data() + (size_t)(c->T + 1) * half;
        for (int s = 0; s <= c->T; ++s) {
            const int row = s ? (s - 1) / c->G : 0, col = s ? (s - 1) % c->G : 0;
            for (int i = 0; i < half; ++i) {
                const int ii = i < quarter ? i : i - quarter;
                const double theta = std::pow((double)m->rope_base, -4.0 * ii / (double)c->dh);
                const double ang = s ? (i < quarter ? row : col) * theta : 0.0;
                cs[(size_t)s * half + i] = (float)std::cos(ang);
                sn[(size_t)s * half + i] = (float)std::sin(ang);
            }
        }
        hbsjd_status st = ensure(c, c->rope, tab.size() * 4);
        if (st != HBSJD_OK) {
            delete c;
            return st;
        }
        e = hipMemcpy(c->rope.p, tab.data(), tab.size() * 4, hipMemcpyHostToDevice);
        if (e != hipSuccess) {
            delete c;
            return fail(HBSJD_EHIP, std::string("hipMemcpy: ") + hipGetErrorString(e));
        }
        *out = c;
        return HBSJD_OK;
    } catch (...) {
        return fail(HBSJD_EINTERNAL, "unexpected host exception in hbsjd_create");
    }
}

void hbsjd_destroy(hbsjd_ctx* ctx) {
    if (!ctx) return;
    (void)hipSetDevice(ctx->device);
    delete ctx;
}

hbsjd_status hbsjd_load_weights(hbsjd_ctx* c, const float* blob, size_t n_floats) {
    try {
        GUARD(c);
        if (!blob) return fail(HBSJD_EINVAL, "blob is NULL");
        if (n_floats != blob_floats(c))
            return fail(HBSJD_EINVAL, "blob has " + std::to_string(n_floats) + " floats, model needs " +
                                          std::to_string(blob_floats(c)));
        const size_t d = c->d, f = c->f, V = c->V, C = c->C, L = c->L, es = c->esz;
        // device layout: embeddings, gains and bias fp32; the GEMM matrices in
        // the compute type (for a bf16 model: rounded to bf16, then held as fp16
        // times a power-of-two scale, see common.h), W1|W3 interleaved by rows
        // (row 2i = W1 row i, row 2i+1 = W3 row i)
        std::vector<size_t> off;
        size_t total = 0;
        auto take = [&](size_t bytes) {
            off.push_back(total);
            total += (bytes + 255) & ~(size_t)255;
        };
        take(V * d * 4);             // tok_emb
        take((C + 1) * d * 4);       // cls_emb
        for (size_t l = 0; l < L; ++l) {
            take(d * 4);             // g_attn
            take(3 * d * d * es);    // wqkv
            take(d * d * es);        // wo
            take(d * 4);             // g_ffn
            take(2 * f * d * es);    // w13
            take(d * f * es);        // w2
        }
        take(d * 4);                 // g_out
        take(V * d * es);            // w_lm
        if (c->m.has_lm_bias) take(V * 4);
        std::vector<unsigned char> host(total, 0);
        // fp32 values (embeddings of a bf16 model rounded to bf16)
        auto put_f32 = [&](size_t dst, const float* src, size_t n, bool round) {
            float* o = reinterpret_cast<float*>(host.data() + dst);
            for (size_t i = 0; i < n; ++i) o[i] = round ? bf16_to_f32(f32_to_bf16(src[i])) : src[i];
        };
        // a GEMM matrix; returns the factor its sums are multiplied by
        auto put_mat = [&](size_t dst, const float* src, size_t n) -> float {
            if (!c->f16) {
                std::memcpy(host.data() + dst, src, n * 4);
                return 1.0f;
            }
            float mx = 0.f;
            for (size_t i = 0; i < n; ++i) mx = std::max(mx, std::fabs(bf16_to_f32(f32_to_bf16(src[i]))));
            // scale 2^e with the largest magnitude in [2^14, 2^15)
            int e = 0;
            if (mx > 0.f) {
                int ex = 0;
                std::frexp(mx, &ex);   // mx in [2^(ex-1), 2^ex)
                e = 15 - ex;
            }
            const float sc = std::ldexp(1.0f, e);
            uint16_t* o = reinterpret_cast<uint16_t*>(host.data() + dst);
            for (size_t i = 0; i < n; ++i) o[i] = f32_to_f16_bits_host(bf16_to_f32(f32_to_bf16(src[i])) * sc);
            return std::ldexp(1.0f, -e);
        };
        const bool rnd = c->f16;
        const float* p = blob;
        size_t k = 0;
        put_f32(off[k++], p, V * d, rnd); p += V * d;
        put_f32(off[k++], p, (C + 1) * d, rnd); p += (C + 1) * d;
        c->s_qkv.assign(L, 1.f); c->s_o.assign(L, 1.f); c->s_13.assign(L, 1.f); c->s_2.assign(L, 1.f);
        for (size_t l = 0; l < L; ++l) {
            put_f32(off[k++], p, d, false); p += d;
            c->s_qkv[l] = put_mat(off[k++], p, 3 * d * d); p += 3 * d * d;
            c->s_o[l] = put_mat(off[k++], p, d * d); p += d * d;
            put_f32(off[k++], p, d, false); p += d;
            {
                const float* w1 = p;
                const float* w3 = p + f * d;
                std::vector<float> il(2 * f * d);
                for (size_t i = 0; i < f; ++i) {
                    std::memcpy(&il[(2 * i) * d], w1 + i * d, d * 4);
                    std::memcpy(&il[(2 * i + 1) * d], w3 + i * d, d * 4);
                }
                c->s_13[l] = put_mat(off[k++], il.data(), 2 * f * d);
                p += 2 * f * d;
            }
            c->s_2[l] = put_mat(off[k++], p, d * f); p += d * f;
        }
        put_f32(off[k++], p, d, false); p += d;
        c->s_lm = put_mat(off[k++], p, V * d); p += V * d;
        if (c->m.has_lm_bias) { put_f32(off[k++], p, V, false); p += V; }
        TRY(ensure(c, c->wbuf, total));
        HIPTRY(c, hipMemcpy(c->wbuf.p, host.data(), total, hipMemcpyHostToDevice));
        char* base = (char*)c->wbuf.p;
        k = 0;
        c->tok_emb = (float*)(base + off[k++]);
        c->cls_emb = (float*)(base + off[k++]);
        c->g_attn.assign(L, nullptr); c->g_ffn.assign(L, nullptr);
        c->wqkv.assign(L, nullptr); c->wo.assign(L, nullptr);
        c->w13.assign(L, nullptr); c->w2.assign(L, nullptr);
        for (size_t l = 0; l < L; ++l) {
            c->g_attn[l] = (float*)(base + off[k++]);
            c->wqkv[l] = base + off[k++];
            c->wo[l] = base + off[k++];
            c->g_ffn[l] = (float*)(base + off[k++]);
            c->w13[l] = base + off[k++];
            c->w2[l] = base + off[k++];
        }
        c->g_out = (float*)(base + off[k++]);
        c->w_lm = base + off[k++];
        c->b_lm = c->m.has_lm_bias ? (float*)(base + off[k++]) : nullptr;
        c->weights = true;
        return HBSJD_OK;
    } catch (...) {
        return fail(HBSJD_EINTERNAL, "unexpected host exception in hbsjd_load_weights");
    }
}

hbsjd_status hbsjd_rollout_begin(hbsjd_ctx* c, const hbsjd_rollout_args* a) {
    try {
        GUARD(c);
        TRY(begin(c, a, nullptr));
        HIPTRY(c, hipStreamSynchronize(c->stream));
        return check_device_error(c);
    } catch (...) {
        return fail(HBSJD_EINTERNAL, "unexpected host exception in hbsjd_rollout_begin");
    }
}

hbsjd_status hbsjd_rollout(hbsjd_ctx* c, const hbsjd_rollout_args* a, hbsjd_rollout_out* o) {
    try {
        GUARD(c);
        if (!o || !o->tokens || !o->counts || !o->rounds)
            return fail(HBSJD_EINVAL, "out.tokens, out.counts and out.rounds are required");
        TRY(begin(c, a, o->counts));
        hipStream_t s = c->stream;
        int rounds = 0;
        // the host stays one round behind the device: it reads A of round r-1
        // while round r is queued; A = 0 means round r-1 (and r) had no work
        for (int r = 0;; ++r) {
            if (r > c->max_rounds + 2) {
                c->poisoned = true;
                return fail(HBSJD_EINTERNAL, "round watchdog: rollout did not finish");
            }
            TRY(launch_round(c));
            HIPTRY(c, hipMemcpyAsync(c->pin + (r & 1), as<int32_t>(c->meta) + kMetaActive, 4,
                                     hipMemcpyDeviceToHost, s));
            HIPTRY(c, hipEventRecord(c->ev[r & 1], s));
            if (r >= 1) {
                HIPTRY(c, hipEventSynchronize(c->ev[(r - 1) & 1]));
                if (c->pin[(r - 1) & 1] == 0) {
                    rounds = r - 1;
                    break;
                }
                c->a_bound = std::min(c->a_bound, (int)c->pin[(r - 1) & 1]);
            }
        }
        HIPTRY(c, hipMemcpyAsync(o->tokens, c->xtok.p, (size_t)c->B * c->T * 4,
                                 hipMemcpyDeviceToDevice, s));
        HIPTRY(c, hipMemcpyAsync(o->counts, c->counts, (size_t)c->max_rounds * c->B * 4,
                                 hipMemcpyDeviceToDevice, s));
        std::vector<int32_t> ah(rounds + 1), mh(rounds + 1);
        int64_t st[4] = {0, 0, 0, 0};
        if (rounds > 0) {
            HIPTRY(c, hipMemcpyAsync(ah.data(), c->a_hist.p, rounds * 4, hipMemcpyDeviceToHost, s));
            HIPTRY(c, hipMemcpyAsync(mh.data(), c->mode_hist.p, rounds * 4, hipMemcpyDeviceToHost, s));
        }
        HIPTRY(c, hipMemcpyAsync(st, c->stats.p, 32, hipMemcpyDeviceToHost, s));
        HIPTRY(c, hipStreamSynchronize(s));
        TRY(check_device_error(c));
        *o->rounds = rounds;
        int64_t rows = 0;
        for (int r = 0; r < rounds; ++r) {
            const int nimg = ah[r] == 0 ? 0 : (mh[r] == 0 ? c->B : ah[r]);
            rows += (int64_t)nimg * c->cfg * (c->W + 1);
        }
        if (o->active_per_round) std::memcpy(o->active_per_round, ah.data(), rounds * 4);
        if (o->mode_per_round) std::memcpy(o->mode_per_round, mh.data(), rounds * 4);
        if (o->stats) {
            o->stats[0] = st[0];
            o->stats[1] = st[1];
            o->stats[2] = st[2];
            o->stats[3] = rows;
        }
        return HBSJD_OK;
    } catch (...) {
        return fail(HBSJD_EINTERNAL, "unexpected host exception in hbsjd_rollout");
    }
}

hbsjd_status hbsjd_round(hbsjd_ctx* c, int32_t exec_mode, int32_t* counts, int32_t* active) {
    try {
        GUARD(c);
        if (!c->have_state) return fail(HBSJD_ESTATE, "no rollout state: call hbsjd_rollout_begin");
        if (exec_mode < HBSJD_EXEC_AUTO || exec_mode > HBSJD_EXEC_COMPACT)
            return fail(HBSJD_EINVAL, "unknown exec_mode");
        if (c->rounds_launched >= c->max_rounds) return fail(HBSJD_ESTATE, "max_rounds reached");
        const int r = c->rounds_launched;
        HIPTRY(c, hipEventRecord(c->ev_user, c->user_stream));
        HIPTRY(c, hipStreamWaitEvent(c->stream, c->ev_user, 0));
        c->exec_mode = exec_mode;
        int32_t em = exec_mode;
        HIPTRY(c, hipMemcpyAsync(as<int32_t>(c->meta) + kMetaExec, &em, 4, hipMemcpyHostToDevice,
                                 c->stream));
        TRY(launch_round(c));
        std::vector<int32_t> cur(c->B);
        if (counts)
            HIPTRY(c, hipMemcpyAsync(counts, c->counts + (size_t)r * c->B, c->B * 4,
                                     hipMemcpyDeviceToHost, c->stream));
        HIPTRY(c, hipMemcpyAsync(cur.data(), c->cursor.p, c->B * 4, hipMemcpyDeviceToHost, c->stream));
        HIPTRY(c, hipStreamSynchronize(c->stream));
        TRY(check_device_error(c));
        int n = 0;
        for (int b = 0; b < c->B; ++b) n += cur[b] < c->T;
        c->a_bound = n;
        if (active) *active = n;
        return HBSJD_OK;
    } catch (...) {
        return fail(HBSJD_EINTERNAL, "unexpected host exception in hbsjd_round");
    }
}

hbsjd_status hbsjd_get_state(hbsjd_ctx* c, int32_t* tokens, int32_t* cursors, int32_t* drafts,
                             float* q_token_prob) {
    try {
        GUARD(c);
        if (!c->have_state) return fail(HBSJD_ESTATE, "no rollout state");
        const int B = c->B, T = c->T, W = c->W;
        const size_t nw = (size_t)B * W;
        std::vector<int32_t> x((size_t)B * T), n(B), dr(nw);
        std::vector<float> qz(nw);
        hipStream_t s = c->stream;
        if (q_token_prob && nw > 0) {
            // the rows the window's reused drafts were drawn from: the prefill's
            // buffer before any round, then the last round's
            const int last = (c->rounds_launched + 1) & 1;
            TRY(ensure(c, c->qz, nw * 4));
            gather_q(as<float>(c->P[last]), as<int32_t>(c->qsrc), as<int32_t>(c->drafts), (int)nw,
                     c->V, c->greedy, as<float>(c->qz), s);
            HIPTRY(c, hipGetLastError());
            HIPTRY(c, hipMemcpyAsync(qz.data(), c->qz.p, nw * 4, hipMemcpyDeviceToHost, s));
        }
        HIPTRY(c, hipMemcpyAsync(x.data(), c->xtok.p, x.size() * 4, hipMemcpyDeviceToHost, s));
        HIPTRY(c, hipMemcpyAsync(n.data(), c->cursor.p, B * 4, hipMemcpyDeviceToHost, s));
        if (nw > 0)
            HIPTRY(c, hipMemcpyAsync(dr.data(), c->drafts.p, nw * 4, hipMemcpyDeviceToHost, s));
        HIPTRY(c, hipStreamSynchronize(s));
        for (int b = 0; b < B; ++b)
            for (int t = n[b]; t < T; ++t) x[(size_t)b * T + t] = 0;
        if (tokens) std::memcpy(tokens, x.data(), x.size() * 4);
        if (cursors) std::memcpy(cursors, n.data(), B * 4);
        if (drafts && nw > 0) std::memcpy(drafts, dr.data(), nw * 4);
        if (q_token_prob && nw > 0) std::memcpy(q_token_prob, qz.data(), nw * 4);
        return HBSJD_OK;
    } catch (...) {
        return fail(HBSJD_EINTERNAL, "unexpected host exception in hbsjd_get_state");
    }
}

hbsjd_status hbsjd_forward(hbsjd_ctx* c, int32_t n_seqs, const int32_t* tokens,
                           const int32_t* lens, const int32_t* labels, float* logits) {
    try {
        GUARD(c);
        if (!c->weights) return fail(HBSJD_ESTATE, "weights not loaded");
        if (n_seqs < 1 || !tokens || !lens || !labels || !logits)
            return fail(HBSJD_EINVAL, "bad forward arguments");
        std::vector<int32_t> simg(n_seqs), ln(n_seqs), lab(n_seqs), row0;
        for (int q = 0; q < n_seqs; ++q) {
            if (lens[q] < 0 || lens[q] > c->T) return fail(HBSJD_EINVAL, "length out of [0, T]");
            if (labels[q] < 0 || labels[q] > c->C) return fail(HBSJD_EINVAL, "label out of [0, n_classes]");
            simg[q] = q;
            ln[q] = lens[q];
            lab[q] = labels[q];
        }
        TRY(forward_core(c, n_seqs, tokens, lab, ln, simg, ln, row0));
        const int rows = row0.back();
        RowBound rb(rows);
        gemm_logits(c->f16, c->hb.p, c->d, c->w_lm, c->s_lm, c->V, c->d,
                    as<int32_t>(c->meta_pf) + kMetaRows, rows, logits, c->b_lm, c->stream);
        HIPTRY(c, hipGetLastError());
        HIPTRY(c, hipStreamSynchronize(c->stream));
        return HBSJD_OK;
    } catch (...) {
        return fail(HBSJD_EINTERNAL, "unexpected host exception in hbsjd_forward");
    }
}

hbsjd_status hbsjd_bikl_rows(const float* logits_s, const float* logits_t, int64_t rows,
                             int32_t V, float* out, void* stream) {
    try {
        if (rows < 0 || rows > INT32_MAX || V < 4 || V > kMaxVocab || V % 4 != 0)
            return fail(HBSJD_EINVAL, "need 0 <= rows < 2^31 and V a multiple of 4 in [4, 16384]");
        if (rows > 0 && (!logits_s || !logits_t || !out)) return fail(HBSJD_EINVAL, "NULL buffer");
        hipStream_t s = (hipStream_t)stream;
        bikl_rows(logits_s, logits_t, (int)rows, V, nullptr, out, s);
        hipError_t e = hipGetLastError();
        if (e == hipSuccess) e = hipStreamSynchronize(s);
        if (e != hipSuccess) return fail(HBSJD_EHIP, std::string("bikl_rows: ") + hipGetErrorString(e));
        return HBSJD_OK;
    } catch (...) {
        return fail(HBSJD_EINTERNAL, "unexpected host exception in hbsjd_bikl_rows");
    }
}

hbsjd_status hbsjd_score_bikl(hbsjd_ctx* student, hbsjd_ctx* teacher, int32_t B,
                              const int32_t* tokens, const int32_t* prefix_len,
                              const int32_t* class_labels, float* per_position, float* loss) {
    try {
        GUARD(teacher);
        GUARD(student);
        if (!student->weights || !teacher->weights) return fail(HBSJD_ESTATE, "weights not loaded");
        if (student == teacher) return fail(HBSJD_EINVAL, "student and teacher must be two contexts");
        if (student->device != teacher->device) return fail(HBSJD_EINVAL, "contexts on different GPUs");
        if (student->T != teacher->T || student->V != teacher->V)
            return fail(HBSJD_EINVAL, "student and teacher need the same grid and vocabulary");
        if (B < 1 || !tokens || !prefix_len || !class_labels || !per_position || !loss)
            return fail(HBSJD_EINVAL, "bad scoring arguments");
        const int T = student->T, C = std::min(student->C, teacher->C);
        // sequences: the images with a generated suffix, teacher-forced over
        // [class, x_1..x_{T-1}]; scored rows: positions k_b..T-1 of each
        std::vector<int32_t> simg, ln, chk(B, 0), lab(B), kk(B), sel, oidx;
        for (int b = 0; b < B; ++b) {
            const int k = prefix_len[b];
            if (k < 0 || k > T) return fail(HBSJD_EINVAL, "prefix_len out of [0, T]");
            if (class_labels[b] < 0 || class_labels[b] >= C)
                return fail(HBSJD_EINVAL, "class label out of [0, n_classes)");
            lab[b] = class_labels[b];
            kk[b] = k;
            if (k == T) continue;
            simg.push_back(b);
            ln.push_back(T - 1);
            chk[b] = T - 1;
        }
        hipStream_t s = student->stream;
        HIPTRY(student, hipEventRecord(student->ev_user, student->user_stream));
        HIPTRY(student, hipStreamWaitEvent(s, student->ev_user, 0));
        HIPTRY(student, hipMemsetAsync(per_position, 0, (size_t)B * T * 4, s));
        const int nq = (int)simg.size();
        if (nq > 0) {
            for (int q = 0; q < nq; ++q)
                for (int p = kk[simg[q]]; p < T; ++p) {
                    sel.push_back(q * T + p);
                    oidx.push_back(simg[q] * T + p);
                }
            const int nsel = (int)sel.size();
            hbsjd_ctx* both[2] = {teacher, student};
            for (hbsjd_ctx* c : both) {
                std::vector<int32_t> row0;
                TRY(forward_core(c, B, tokens, lab, chk, simg, ln, row0));
                TRY(ensure(c, c->lm_idx, (size_t)nsel * 4));
                TRY(ensure(c, c->score_logits, (size_t)nsel * c->V * 4));
                HIPTRY(c, hipMemcpyAsync(c->lm_idx.p, sel.data(), (size_t)nsel * 4,
                                         hipMemcpyHostToDevice, c->stream));
                int32_t* mp = as<int32_t>(c->meta_pf);
                HIPTRY(c, hipMemcpyAsync(mp + kMetaActive, &nsel, 4, hipMemcpyHostToDevice, c->stream));
                RowBound rb(nsel);
                rmsnorm(c->f16, as<float>(c->h), as<int32_t>(c->lm_idx), mp + kMetaActive, nsel,
                        c->g_out, c->m.rms_eps, c->d, c->hb.p, c->stream);
                gemm_logits(c->f16, c->hb.p, c->d, c->w_lm, c->s_lm, c->V, c->d, mp + kMetaActive, nsel,
                            as<float>(c->score_logits), c->b_lm, c->stream);
                HIPTRY(c, hipGetLastError());
            }
            if (!teacher->ev_done)
                HIPTRY(teacher, hipEventCreateWithFlags(&teacher->ev_done, hipEventDisableTiming));
            HIPTRY(teacher, hipEventRecord(teacher->ev_done, teacher->stream));
            HIPTRY(student, hipStreamWaitEvent(s, teacher->ev_done, 0));
            TRY(ensure(student, student->score_idx, (size_t)nsel * 4));
            TRY(ensure(student, student->score_k, (size_t)B * 4));
            HIPTRY(student, hipMemcpyAsync(student->score_idx.p, oidx.data(), (size_t)nsel * 4,
                                           hipMemcpyHostToDevice, s));
            HIPTRY(student, hipMemcpyAsync(student->score_k.p, kk.data(), (size_t)B * 4,
                                           hipMemcpyHostToDevice, s));
            {
                Timed tm(student, HBSJD_K_BIKL);
                bikl_rows(as<float>(student->score_logits), as<float>(teacher->score_logits), nsel,
                          student->V, as<int32_t>(student->score_idx), per_position, s);
            }
            bikl_mean(per_position, as<int32_t>(student->score_k), B, T, loss, s);
        } else {
            HIPTRY(student, hipMemsetAsync(loss, 0, (size_t)B * 4, s));
        }
        HIPTRY(student, hipGetLastError());
        HIPTRY(student, hipStreamSynchronize(s));   // also keeps the host staging alive
        return HBSJD_OK;
    } catch (...) {
        return fail(HBSJD_EINTERNAL, "unexpected host exception in hbsjd_score_bikl");
    }
}

// Fixed device workspace of hbsjd_transform_rows_noalloc: the per-row metadata
// of up to HBSJD_NOALLOC_MAX_ROWS rows. Every GPU the library runs on holds its
// own copy for the life of the process. Host code never passes this name to a
// kernel or a copy (on the host it is only a stand-in for the symbol); it uses
// the device address that hipGetSymbolAddress returns for the current device.
static __device__ __align__(256) int32_t scratch[2 * HBSJD_NOALLOC_MAX_ROWS + kMetaCount];

namespace {
std::mutex g_scratch_mu;
std::vector<int32_t*> g_scratch_ptr;   // per device: the address of its `scratch`

// the current device's copy of `scratch`, looked up once per device
hbsjd_status static_scratch(int32_t** out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return fail(HBSJD_EHIP, std::string("hipGetDevice: ") + hipGetErrorString(e));
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if ((int)g_scratch_ptr.size() <= dev) g_scratch_ptr.resize(dev + 1, nullptr);
    if (!g_scratch_ptr[dev]) {
        void* ptr = nullptr;
        e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !ptr)
            return fail(HBSJD_EHIP, std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(e));
        g_scratch_ptr[dev] = static_cast<int32_t*>(ptr);
    }
    *out = g_scratch_ptr[dev];
    return HBSJD_OK;
}

hbsjd_status check_transform_rows(int32_t rows, int32_t V, const float* logits, int32_t cfg,
                                  float cfg_scale, const float* temperature, int32_t top_k,
                                  const int32_t* position, const float* p, const int32_t* argmax,
                                  const int32_t* draw) {
    if (rows < 1) return fail(HBSJD_EINVAL, "need rows >= 1");
    if (V < 4 || V > kMaxVocab || V % 4) return fail(HBSJD_EINVAL, "need V a multiple of 4 in [4, 16384]");
    if (cfg != 1 && cfg != 2) return fail(HBSJD_EINVAL, "cfg must be 1 or 2");
    if (cfg == 2 && !std::isfinite(cfg_scale)) return fail(HBSJD_EINVAL, "cfg_scale not finite");
    if (top_k < 0) return fail(HBSJD_EINVAL, "top_k < 0");
    if (!logits || !temperature || !position || !p || !argmax || !draw)
        return fail(HBSJD_EINVAL, "NULL buffer");
    if (cfg == 2 && (const void*)p == (const void*)logits)
        return fail(HBSJD_EINVAL, "p may alias logits only without guidance");
    return HBSJD_OK;
}

hbsjd_status finish_transform_rows(const int32_t* meta, hipStream_t s) {
    int32_t err = 0;
    hipError_t e = hipGetLastError();
    if (e == hipSuccess) e = hipMemcpyAsync(&err, meta + kMetaError, 4, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return fail(HBSJD_EHIP, std::string("transform_rows: ") + hipGetErrorString(e));
    if (err & kErrNanLogit) return fail(HBSJD_EINVAL, "a logit is NaN");
    return HBSJD_OK;
}
}  // namespace

hbsjd_status hbsjd_transform_rows(int32_t rows, int32_t V, const float* logits, int32_t cfg,
                                  float cfg_scale, const float* temperature, int32_t top_k,
                                  uint64_t seed, const int32_t* position, float* p,
                                  int32_t* argmax, int32_t* draw, void* stream) {
    try {
        TRY(check_transform_rows(rows, V, logits, cfg, cfg_scale, temperature, top_k, position, p,
                                 argmax, draw));
        hipStream_t s = (hipStream_t)stream;
        int32_t* scratch = nullptr;
        hipError_t e = hipMalloc((void**)&scratch, transform_rows_scratch(rows) * 4);
        if (e != hipSuccess) return fail(HBSJD_ENOMEM, "transform_rows scratch");
        transform_rows(rows, V, logits, cfg, cfg_scale, temperature, top_k, seed, position, p,
                       argmax, draw, scratch, s);
        const hbsjd_status st = finish_transform_rows(scratch + 2 * (size_t)rows, s);
        (void)hipFree(scratch);
        return st;
    } catch (...) {
        return fail(HBSJD_EINTERNAL, "unexpected host exception in hbsjd_transform_rows");
    }
}

hbsjd_status hbsjd_transform_rows_noalloc(int32_t rows, int32_t V, const float* logits,
                                          int32_t cfg, float cfg_scale, const float* temperature,
                                          int32_t top_k, uint64_t seed, const int32_t* position,
                                          float* p, int32_t* argmax, int32_t* draw, void* stream) {
    try {
        if (rows > HBSJD_NOALLOC_MAX_ROWS)
            return fail(HBSJD_EINVAL, "rows exceeds HBSJD_NOALLOC_MAX_ROWS (65536)");
        TRY(check_transform_rows(rows, V, logits, cfg, cfg_scale, temperature, top_k, position, p,
                                 argmax, draw));
        int32_t* ws = nullptr;
        TRY(static_scratch(&ws));
        hipStream_t s = (hipStream_t)stream;
        transform_rows(rows, V, logits, cfg, cfg_scale, temperature, top_k, seed, position, p,
                       argmax, draw, ws, s);
        return finish_transform_rows(ws + 2 * (size_t)rows, s);
    } catch (...) {
        return fail(HBSJD_EINTERNAL, "unexpected host exception in hbsjd_transform_rows_noalloc");
    }
}

hbsjd_status hbsjd_verify_probs(int32_t B, int32_t W, int32_t V, const float* p, const float* q,
                                const int32_t* drafts, const float* u_acc, const float* u_res,
                                int32_t* counts, int32_t* tokens, void* stream) {
    try {
        if (B < 1 || W < 1 || V < 4 || V > kMaxVocab || V % 4)
            return fail(HBSJD_EINVAL, "need B >= 1, W >= 1, V a multiple of 4 in [4, 16384]");
        if (!p || !q || !drafts || !u_acc || !u_res || !counts || !tokens)
            return fail(HBSJD_EINVAL, "NULL buffer");
        hipStream_t s = (hipStream_t)stream;
        verify_probs(B, W, V, p, q, drafts, u_acc, u_res, counts, tokens, s);
        hipError_t e = hipGetLastError();
        if (e == hipSuccess) e = hipStreamSynchronize(s);
        if (e != hipSuccess) return fail(HBSJD_EHIP, std::string("verify_probs: ") + hipGetErrorString(e));
        return HBSJD_OK;
    } catch (...) {
        return fail(HBSJD_EINTERNAL, "unexpected host exception in hbsjd_verify_probs");
    }
}

hbsjd_status hbsjd_philox(uint64_t seed, int32_t n, const uint32_t* bt, uint32_t* out, void* stream) {
    try {
        if (n < 0 || (n > 0 && (!bt || !out))) return fail(HBSJD_EINVAL, "bad philox arguments");
        hipStream_t s = (hipStream_t)stream;
        philox_fill(seed, n, bt, out, s);
        hipError_t e = hipGetLastError();
        if (e == hipSuccess) e = hipStreamSynchronize(s);
        if (e != hipSuccess) return fail(HBSJD_EHIP, std::string("philox: ") + hipGetErrorString(e));
        return HBSJD_OK;
    } catch (...) {
        return fail(HBSJD_EINTERNAL, "unexpected host exception in hbsjd_philox");
    }
}

hbsjd_status hbsjd_mfma_probe(int32_t workgroups, int32_t iters, float* sink, void* stream) {
    try {
        if (workgroups < 1 || iters < 1 || !sink) return fail(HBSJD_EINVAL, "bad mfma probe arguments");
        hipStream_t s = (hipStream_t)stream;
        mfma_probe(workgroups, iters, sink, s);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return fail(HBSJD_EHIP, std::string("mfma probe: ") + hipGetErrorString(e));
        return HBSJD_OK;
    } catch (...) {
        return fail(HBSJD_EINTERNAL, "unexpected host exception in hbsjd_mfma_probe");
    }
}

hbsjd_status hbsjd_profile_start(hbsjd_ctx* c, uint32_t class_mask) {
    try {
        GUARD(c);
        prof_resolve(c);
        for (int k = 0; k < HBSJD_K_COUNT; ++k) {
            c->prof_ms[k] = 0.0;
            c->prof_n[k] = 0;
            c->prof_seen[k] = 0;
        }
        c->prof_mask = class_mask & ((1u << HBSJD_K_COUNT) - 1);
        return HBSJD_OK;
    } catch (...) {
        return fail(HBSJD_EINTERNAL, "unexpected host exception in hbsjd_profile_start");
    }
}

hbsjd_status hbsjd_profile_sample(hbsjd_ctx* c, int32_t every) {
    try {
        GUARD(c);
        if (every < 1) return fail(HBSJD_EINVAL, "profile sample interval must be >= 1");
        c->prof_every = every;
        return HBSJD_OK;
    } catch (...) {
        return fail(HBSJD_EINTERNAL, "unexpected host exception in hbsjd_profile_sample");
    }
}

hbsjd_status hbsjd_profile_read(hbsjd_ctx* c, double* total_ms, int64_t* launches) {
    try {
        GUARD(c);
        HIPTRY(c, hipStreamSynchronize(c->stream));
        prof_resolve(c);
        for (int k = 0; k < HBSJD_K_COUNT; ++k) {
            if (total_ms) total_ms[k] = c->prof_ms[k];
            if (launches) launches[k] = c->prof_n[k];
        }
        return HBSJD_OK;
    } catch (...) {
        return fail(HBSJD_EINTERNAL, "unexpected host exception in hbsjd_profile_read");
    }
}

hbsjd_status hbsjd_calibrate_gamma(hbsjd_ctx* c, int32_t batch, int32_t window, int32_t* gamma) {
    try {
        GUARD(c);
        if (!gamma) return fail(HBSJD_EINVAL, "gamma is NULL");
        if (!c->weights) return fail(HBSJD_ESTATE, "weights not loaded");
        if (batch < 1 || window < 1 || window > 64)
            return fail(HBSJD_EINVAL, "need batch >= 1 and window in [1, 64]");
        hipStream_t s = c->stream;
        const int B = batch, T = c->T, k = T / 2;
        // data-independent state: every image halfway through an all-zero
        // prefix of class 0; only the verifier forward is timed
        TRY(ensure(c, c->calib_tok, (size_t)B * T * 4));
        HIPTRY(c, hipMemsetAsync(c->calib_tok.p, 0, (size_t)B * T * 4, s));
        std::vector<int32_t> plen(B, k), lab(B, 0), cur(B);
        std::vector<float> tau(B, 1.f);
        hbsjd_rollout_args a{};
        a.batch = B;
        a.prefix_tokens = as<int32_t>(c->calib_tok);
        a.prefix_len = plen.data();
        a.class_labels = lab.data();
        a.temperature = tau.data();
        a.window = window;
        a.history = 24;
        a.verify_mode = HBSJD_VERIFY_PROB;
        a.exec_mode = HBSJD_EXEC_FULL;
        a.gamma = 0;
        a.max_rounds = T;
        TRY(begin(c, &a, nullptr));
        c->have_state = false;   // the synthetic state is not a rollout
        hipEvent_t e0, e1;
        HIPTRY(c, hipEventCreate(&e0));
        HIPTRY(c, hipEventCreate(&e1));
        auto time_mode = [&](int exec, float* us) -> hbsjd_status {
            c->exec_mode = exec;           // with a_bound, the row bound of the timed rounds
            int32_t hdr[2] = {-1, exec};   // round index, exec mode
            HIPTRY(c, hipMemcpyAsync(as<int32_t>(c->meta) + kMetaRound, &hdr[0], 4, hipMemcpyHostToDevice, s));
            HIPTRY(c, hipMemcpyAsync(as<int32_t>(c->meta) + kMetaExec, &hdr[1], 4, hipMemcpyHostToDevice, s));
            enqueue_round(c, 0, false);   // warm-up
            constexpr int kReps = 5;
            HIPTRY(c, hipEventRecord(e0, s));
            for (int r = 0; r < kReps; ++r) enqueue_round(c, r & 1, false);
            HIPTRY(c, hipEventRecord(e1, s));
            HIPTRY(c, hipEventSynchronize(e1));
            float ms = 0.f;
            HIPTRY(c, hipEventElapsedTime(&ms, e0, e1));
            *us = 1000.f * ms / kReps;
            return HBSJD_OK;
        };
        int best = 0;
        std::vector<int> cand;
        for (int A = 1; A < B; A *= 2) cand.push_back(A);
        cand.push_back(B);
        hbsjd_status st = HBSJD_OK;
        // Eq. 6: Compact iff A <= gamma. "No slower" allows 2% of timing
        // noise; with every image active (A = B) the two modes run the same
        // rows, so that case is a tie and is not timed.
        for (int A : cand) {
            if (A == B) {
                if (best == cand[cand.size() > 1 ? cand.size() - 2 : 0] || B == 1) best = B;
                break;
            }
            for (int b = 0; b < B; ++b) cur[b] = b < A ? k : T;
            HIPTRY(c, hipMemcpyAsync(c->cursor.p, cur.data(), B * 4, hipMemcpyHostToDevice, s));
            c->a_bound = A;
            float t_full = 0.f, t_compact = 0.f;
            if ((st = time_mode(HBSJD_EXEC_FULL, &t_full)) != HBSJD_OK) break;
            if ((st = time_mode(HBSJD_EXEC_COMPACT, &t_compact)) != HBSJD_OK) break;
            if (t_compact <= 1.02f * t_full) best = A;
        }
        (void)hipEventDestroy(e0);
        (void)hipEventDestroy(e1);
        TRY(st);
        HIPTRY(c, hipGetLastError());
        c->gamma_cal = best;
        *gamma = best;
        return HBSJD_OK;
    } catch (...) {
        return fail(HBSJD_EINTERNAL, "unexpected host exception in hbsjd_calibrate_gamma");
    }
}

}  // extern "C"
