// Host-side launchers of the library's kernels (internal interface).
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <cstdint>
#include <vector>

#include "common.h"

namespace hbsjd {

// Optional kernel timing: while a caller has the per-thread slot armed, the
// launches through launch() carry the events in their own dispatches
// (hipExtLaunchKernelGGL): the first one the start event, every one the stop
// event, so the pair spans the kernels of the armed region (one GEMM may be
// two launches, of which one finds nothing to do) and nothing else.
struct LaunchEvents {
    hipEvent_t start = nullptr;
    hipEvent_t stop = nullptr;
    bool used = false;
};
LaunchEvents* launch_events();

template <typename K, typename... Args>
inline void launch(K kernel, dim3 grid, dim3 block, uint32_t shmem, hipStream_t s, Args... args) {
    LaunchEvents* ev = launch_events();
    if (ev->start) {
        hipExtLaunchKernelGGL(kernel, grid, block, shmem, s, ev->used ? nullptr : ev->start,
                              ev->stop, 0u, args...);
        ev->used = true;
    } else {
        hipLaunchKernelGGL(kernel, grid, block, shmem, s, args...);
    }
}

// The paged KV cache of one layer is an array of pages of 64 slots; page p
// holds, for every head h, K as [64 slots][head_dim] at
// (p * 2 * heads + h) * 64 * head_dim and V transposed as [head_dim][64 slots]
// at (p * 2 * heads + heads + h) * 64 * head_dim. A sequence's page table maps
// its tile j (positions 64 j .. 64 j + 63) to a page.

// Per-row metadata of a verifier (or prefill) forward.
struct RowMeta {
    const int32_t* tok;   // token id, or -(1 + class) for the class embedding
    const int32_t* pos;   // sequence position
    const int32_t* kv;    // page * 64 + slot of the row's KV entry
    const int32_t* seq;   // sequence (image * cfg + branch)
};

// Attention segments: consecutive rows of one sequence at consecutive positions.
struct Segments {
    const int32_t* seq;
    const int32_t* row0;
    const int32_t* nrows;
    const int32_t* pos0;
    const int32_t* pages;   // [segment][max_pages]: KV page of each 64-key tile of its sequence
};
// pages[q][j] = ptab[seq[q]][j] for the nseg segments (host-built segment lists)
void seg_pages(const int32_t* seq, int nseg, const int32_t* ptab, int max_pages, int32_t* pages,
               hipStream_t s);

// ---------------------------------------------------------------- GEMM
// C[M x N] = A[M x K] . W[N x K]^T with a fused epilogue. M is read from
// m_dev (clamped to m_cap) when m_dev is not null; the grid covers m_cap rows.

struct QkvArgs {
    void* q;              // [M][d] activation dtype
    void* kv;             // layer base of the KV pool
    const int32_t* pos;
    const int32_t* kvslot;
    const float* rope_cos;   // [(T+1)][dh/2]
    const float* rope_sin;
    int d, heads, head_dim, T;
};

// With f16, A and W are fp16 and the sums are multiplied by wscale (the
// inverse of the power-of-two scale the weights are held with); the fp32 path
// ignores wscale.
void gemm_qkv(bool f16, const void* A, int lda, const void* W, float wscale, int N, int K,
              const int* m_dev, int m_cap, const QkvArgs& e, hipStream_t s);
// once per process before any launch (the wide GEMM's LDS allowance)
hipError_t gemm_setup();
// An upper bound, known on the host, of the rows present in this thread's
// following launches whose row count is read on the device (-1: none). With
// one, such a product launches the single kernel that suits the bound instead
// of two kernels that choose between themselves on the device. Any kernel is
// correct for any row count up to the launch's cap, so a bound that is too
// small only costs speed.
void gemm_row_bound(int rows);
// The kernels of one product (kGemmWide alone, kGemm128 or kGemm64 alone, or
// kGemmPair | the smaller-tile kernel; kGemmDeep marks the 4-stage 64 x 64
// variant), recorded with its shape by every product with a device row count
// while a log is set (null: none). A round captured under one row bound
// serves a smaller bound while gemm_plan() gives every product it recorded
// the same kernels under that bound (its launches are sized for the larger).
enum { kGemmWide = 4, kGemm128 = 1, kGemm64 = 2, kGemmPair = 8, kGemmDeep = 16 };
struct GemmPlan {
    int N, K, m_cap, splits;
    bool wide_ok;
    int kernels;
};
void gemm_plan_log(std::vector<GemmPlan>* log);
int gemm_plan(const GemmPlan& p, int row_bound);
// reads HBSJD_ATTN_KERNEL ("seq" / "split": one attention kernel for every launch)
void attention_setup();
// MFMA calibration kernel: workgroups x 4 wavefronts x iters x 8 MFMAs (16384 flops each)
void mfma_probe(int workgroups, int iters, float* sink, hipStream_t s);
// split-K partial sums part[split][m_cap][N] (tag 0: O projection, 1: W2);
// split_for() is the split count the host must size `part` for
int split_for(int m_cap, int N, int K);
void gemm_partial(bool f16, int tag, const void* A, int lda, const void* W, float wscale, int N,
                  int K, const int* m_dev, int m_cap, int splits, float* part, hipStream_t s);
// MFMA path with one K part: h[m_cap][N] += A W^T in the epilogue (tag as above)
void gemm_residual(int tag, const void* A, int lda, const void* W, float wscale, int N, int K,
                   const int* m_dev, int m_cap, float* h, hipStream_t s);
void gemm_swiglu(bool f16, const void* A, int lda, const void* W, float wscale, int N, int K,
                 const int* m_dev, int m_cap, void* act, hipStream_t s);
void gemm_logits(bool f16, const void* A, int lda, const void* W, float wscale, int N, int K,
                 const int* m_dev, int m_cap, float* out, const float* bias, hipStream_t s);

// ---------------------------------------------------------------- attention
void attention(bool f16, const void* q, void* o, int d, int heads, int head_dim,
               const void* kv_layer, const int32_t* ptab, int max_pages, const Segments& seg,
               const int* nseg_dev, int nseg_cap, int max_rows_per_seg, const RowMeta& rows,
               const int* nrows_dev, int nrows_cap, hipStream_t s);

// ---------------------------------------------------------------- row ops
// the embedding tables are fp32 on both paths
void embed_norm(bool f16, const RowMeta& rows, const int* nrows_dev, int nrows_cap,
                const float* tok_emb, const float* cls_emb, const float* gain, float eps, int d,
                float* h, void* hb, hipStream_t s);
void rmsnorm(bool f16, const float* h, const int32_t* src_idx, const int* nrows_dev,
             int nrows_cap, const float* gain, float eps, int d, void* hb, hipStream_t s);
// h += sum over splits (in split order) of part[split][m_cap][d]; then
// hb = RMSNorm(h) * gain (hb may be null). With splits = 0 the sum is already
// in h (gemm_residual) and only hb is written.
void reduce_residual_norm(bool f16, const float* part, int splits, int m_cap, float* h,
                          const int* nrows_dev, const float* gain, float eps, int d, void* hb,
                          hipStream_t s);

struct RoundSetupArgs {
    int B, W, T, cfg, C, max_pages, max_rounds;   // gamma and exec mode come from meta
    const int32_t* cursor;
    const int32_t* drafts;
    const int32_t* xtok;
    const int32_t* labels;
    const int32_t* ptab;
    int32_t* slot_img;
    int32_t* active_list;
    int32_t* row_tok;
    int32_t* row_pos;
    int32_t* row_kv;
    int32_t* row_seq;
    int32_t* seg_seq;
    int32_t* seg_row0;
    int32_t* seg_nrows;
    int32_t* seg_pos0;
    int32_t* meta;
    int32_t* a_hist;
    int32_t* mode_hist;
    int32_t* seg_pages;
    int32_t* win_end;   // batch-synchronous windows: [B] end of each image's window; null otherwise
};
void round_setup(const RoundSetupArgs& a, hipStream_t s);

struct PrefillRowsArgs {
    int n_seq, T, cfg, C, max_pages, total_rows;
    const int32_t* seq_row0;     // [n_seq + 1]
    const int32_t* seq_img;      // [n_seq]
    const int32_t* seq_branch;   // [n_seq]
    const int32_t* prefix;       // device [B][T]
    const int32_t* labels;       // device [B]
    const int32_t* ptab;
    int32_t* row_tok;
    int32_t* row_pos;
    int32_t* row_kv;
    int32_t* row_seq;
};
void prefill_rows(const PrefillRowsArgs& a, hipStream_t s);
void check_prefix(const int32_t* prefix, const int32_t* len, int B, int T, int V, int32_t* err,
                  hipStream_t s);
void philox_fill(uint64_t seed, int n, const uint32_t* bt, uint32_t* out, hipStream_t s);

// ---------------------------------------------------------------- sampler
struct TransformArgs {
    const float* logits;     // forward rows [rows][V]
    float* p;                // distribution rows [out][V] (may equal logits without CFG)
    int32_t* amax;           // [out]
    int32_t* samp;           // [out] each row's draw for the position it predicts (-1 past T)
    const int32_t* slot_img;
    const int32_t* cursor;   // [B]: row i of image b predicts position cursor[b] + i + 1
    const float* temperature;   // [B]
    int rows_per_slot, cfg, V, top_k, T;
    float cfg_scale;
    const int* nout_dev;
    int nout_cap;
    int32_t* meta;
};
void transform(const TransformArgs& a, hipStream_t s);

struct VerifyArgs {
    int B, W, T, H, V, greedy, prefill, rows_per_slot, max_rounds;   // seed comes from meta
    const float* p;          // this round's distribution rows
    const int32_t* amax;
    const int32_t* samp;     // this round's draft candidates (from the transform)
    const float* p_prev;     // previous round's rows (proposals)
    const int32_t* slot_img;
    const int* nimg_dev;
    int nimg_cap;
    int32_t* cursor;
    int32_t* xtok;
    int32_t* drafts;
    int32_t* qsrc;
    int32_t* counts;         // [max_rounds][B] or null
    int64_t* stats;          // [4]
    int32_t* meta;
    int ar = 0;              // cached-AR rounds: commit one draw of each image's single row
    const int32_t* win_end = nullptr;   // batch-synchronous windows: verify up to win_end[b]
};
void verify_commit(const VerifyArgs& a, hipStream_t s);
// q[i] for the state export: p(z) of a reused draft's source row, 1 for a
// history draft or in greedy mode, 0 without a draft
void gather_q(const float* P, const int32_t* qsrc, const int32_t* drafts, int n, int V,
              int greedy, float* q, hipStream_t s);

// The transform of caller rows (row r = image r at position pos[r], clamped to
// [0, kRowPosMax]): logits [rows][cfg][V]; outputs p [rows][V], amax and draw
// [rows]. `scratch` holds transform_rows_scratch(rows) int32 words.
constexpr int kRowPosMax = 1 << 30;
inline size_t transform_rows_scratch(int rows) { return 2 * (size_t)rows + kMetaCount; }
void transform_rows(int rows, int V, const float* logits, int cfg, float cfg_scale,
                    const float* temperature, int top_k, uint64_t seed, const int32_t* pos,
                    float* p, int32_t* amax, int32_t* draw, int32_t* scratch, hipStream_t s);

// ---------------------------------------------------------------- teacher scoring
// per row r: D_biKL(softmax(ls[r]), softmax(lt[r])) into out[out_idx ? out_idx[r] : r]
void bikl_rows(const float* ls, const float* lt, int rows, int V, const int32_t* out_idx,
               float* out, hipStream_t s);
// loss[b] = mean of per[b][t-1] over t = k[b]+1..T (0 when k[b] = T)
void bikl_mean(const float* per, const int32_t* k, int B, int T, float* loss, hipStream_t s);

void verify_probs(int B, int W, int V, const float* p, const float* q, const int32_t* drafts,
                  const float* u_acc, const float* u_res, int32_t* counts, int32_t* tokens,
                  hipStream_t s);

}  // namespace hbsjd
