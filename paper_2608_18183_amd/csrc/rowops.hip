// Row bookkeeping of the rollout: per-round active compaction and execution
// mode (Sec. 4.3, Eq. 6), verifier-row assembly (last committed token followed
// by the draft window at per-image positions and KV slots, Sec. 4.2), prefill
// rows, the embedding gather, and RMSNorm.
#include <type_traits>

#include "common.h"
#include "launch.h"

namespace hbsjd {

// ---------------------------------------------------------------- round set-up
// One workgroup. Prefix-scan of active flags (n_b < T) gives A and the ordered
// list of active images; Full processes every image (finished ones computed
// and discarded), Compact only the active list. Then writes the row metadata
// of the chosen images: row (slot, branch, i) holds position n_b + i with token
// x_{n_b} (class token when n_b = 0) for i = 0 and draft i otherwise.
__global__ __launch_bounds__(1024) void k_round_setup(RoundSetupArgs a) {
    __shared__ int warp_tot[16];
    __shared__ int s_base;
    const int t = threadIdx.x, lane = t & 63, wv = t >> 6;
    if (t == 0) s_base = 0;
    // batch-synchronous windows: the batch moves on to the next window once no
    // active image has drafts of its current one left to verify. Every reader
    // derives the new end from the old one; the owners store it at the end.
    int pend = 0;
    if (a.win_end)
        for (int b = t; b < a.B; b += 1024) pend |= a.cursor[b] < min(a.win_end[b], a.T) ? 1 : 0;
    const bool advance = a.win_end && !__syncthreads_or(pend);
    auto window_end = [&](int b) {
        if (!a.win_end) return a.T;
        const int e = a.win_end[b];
        return advance ? min(e + a.W, a.T) : e;
    };
    __syncthreads();
    for (int c0 = 0; c0 < a.B; c0 += 1024) {
        const int b = c0 + t;
        const int act = (b < a.B && a.cursor[b] < a.T) ? 1 : 0;
        // inclusive scan inside the wave
        int x = act;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            const int y = __shfl_up(x, o, 64);
            if (lane >= o) x += y;
        }
        if (lane == 63) warp_tot[wv] = x;
        __syncthreads();
        int before = s_base;
        for (int k = 0; k < wv; ++k) before += warp_tot[k];
        if (act) a.active_list[before + x - 1] = b;
        __syncthreads();
        if (t == 0) {
            int s = s_base;
            for (int k = 0; k < 16; ++k) s += warp_tot[k];
            s_base = s;
        }
        __syncthreads();
    }
    const int A = s_base;
    const int exec_mode = a.meta[kMetaExec];
    int mode;
    if (exec_mode == 1) mode = 0;
    else if (exec_mode == 2) mode = 1;
    else mode = A > a.meta[kMetaGamma] ? 0 : 1;
    const int nimg = A == 0 ? 0 : (mode == 0 ? a.B : A);
    const int R = a.W + 1;
    const int rows = nimg * a.cfg * R;
    for (int s = t; s < nimg; s += 1024) a.slot_img[s] = mode == 0 ? s : a.active_list[s];
    __syncthreads();
    for (int r = t; r < rows; r += 1024) {
        const int s = r / (a.cfg * R);
        const int rem = r - s * a.cfg * R;
        const int br = rem / R, i = rem - br * R;
        const int b = a.slot_img[s];
        int n = a.cursor[b];
        n = n > a.T ? a.T : n;
        const int We = max(min(a.W, window_end(b) - n), 0);
        const int seq = b * a.cfg + br;
        const int pos = n + i;
        int tok;
        if (i == 0)
            tok = n == 0 ? -(1 + (br == 0 ? a.labels[b] : a.C)) : a.xtok[(size_t)b * a.T + n - 1];
        else
            tok = i <= We ? a.drafts[(size_t)b * a.W + i - 1] : 0;
        a.row_tok[r] = tok;
        a.row_pos[r] = pos;
        a.row_seq[r] = seq;
        a.row_kv[r] = a.ptab[(size_t)seq * a.max_pages + (pos >> 6)] * 64 + (pos & 63);
    }
    for (int q = t; q < nimg * a.cfg; q += 1024) {
        const int s = q / a.cfg, br = q - s * a.cfg;
        const int b = a.slot_img[s];
        int n = a.cursor[b];
        n = n > a.T ? a.T : n;
        const int seq = b * a.cfg + br;
        a.seg_seq[q] = seq;
        a.seg_row0[q] = q * R;
        a.seg_nrows[q] = R;
        a.seg_pos0[q] = n;
        for (int j = 0; j < a.max_pages; ++j)
            a.seg_pages[(size_t)q * a.max_pages + j] = a.ptab[(size_t)seq * a.max_pages + j];
    }
    if (t == 0) {
        const int round = a.meta[kMetaRound] + 1;
        a.meta[kMetaRound] = round;
        a.meta[kMetaRows] = rows;
        a.meta[kMetaOutRows] = nimg * R;
        a.meta[kMetaImgs] = nimg;
        a.meta[kMetaSegs] = nimg * a.cfg;
        a.meta[kMetaActive] = A;
        a.meta[kMetaMode] = mode;
        if (round < a.max_rounds) {
            a.a_hist[round] = A;
            a.mode_hist[round] = mode;
        } else if (A > 0) {
            atomicOr(&a.meta[kMetaError], (int)kErrRoundOverflow);
        }
    }
    if (advance) {
        __syncthreads();   // every read of the old ends is done
        for (int b = t; b < a.B; b += 1024) a.win_end[b] = min(a.win_end[b] + a.W, a.T);
    }
}

void round_setup(const RoundSetupArgs& a, hipStream_t s) {
    launch(k_round_setup, dim3(1), dim3(1024), 0, s, a);
}

__global__ void k_seg_pages(const int32_t* seq, int nseg, const int32_t* ptab, int maxp,
                            int32_t* pages) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= nseg * maxp) return;
    const int q = i / maxp, j = i - q * maxp;
    pages[i] = ptab[(size_t)seq[q] * maxp + j];
}

void seg_pages(const int32_t* seq, int nseg, const int32_t* ptab, int max_pages, int32_t* pages,
               hipStream_t s) {
    const int n = nseg * max_pages;
    if (n <= 0) return;
    launch(k_seg_pages, dim3((n + 255) / 256), dim3(256), 0, s, seq, nseg, ptab, max_pages, pages);
}

// ---------------------------------------------------------------- prefill rows
// row r of sequence q (image b, branch br) is position r - seq_row0[q]: the
// class token at 0, prefix token x_p at p >= 1.
__global__ void k_prefill_rows(PrefillRowsArgs a) {
    const int r = blockIdx.x * blockDim.x + threadIdx.x;
    if (r >= a.total_rows) return;
    int lo = 0, hi = a.n_seq;   // find q with seq_row0[q] <= r < seq_row0[q+1]
    while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (a.seq_row0[mid] <= r) lo = mid; else hi = mid;
    }
    const int q = lo;
    const int b = a.seq_img[q], br = a.seq_branch[q];
    const int pos = r - a.seq_row0[q];
    const int seq = b * a.cfg + br;
    a.row_tok[r] = pos == 0 ? -(1 + (br == 0 ? a.labels[b] : a.C))
                            : a.prefix[(size_t)b * a.T + pos - 1];
    a.row_pos[r] = pos;
    a.row_seq[r] = seq;
    a.row_kv[r] = a.ptab[(size_t)seq * a.max_pages + (pos >> 6)] * 64 + (pos & 63);
}

void prefill_rows(const PrefillRowsArgs& a, hipStream_t s) {
    if (a.total_rows <= 0) return;
    launch(k_prefill_rows, dim3((a.total_rows + 255) / 256), dim3(256), 0, s, a);
}

__global__ void k_check_prefix(const int32_t* prefix, const int32_t* len, int B, int T, int V,
                               int32_t* err) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= B * T) return;
    const int b = i / T, t = i - b * T;
    if (t < len[b]) {
        const int v = prefix[i];
        if (v < 0 || v >= V) atomicOr(err, (int)kErrBadToken);
    }
}

void check_prefix(const int32_t* prefix, const int32_t* len, int B, int T, int V, int32_t* err,
                  hipStream_t s) {
    const int n = B * T;
    if (n <= 0) return;
    launch(k_check_prefix, dim3((n + 255) / 256), dim3(256), 0, s, prefix, len, B, T,
                       V, err);
}

// ---------------------------------------------------------------- norms
// RMSNorm(x) * g = x * (1 / sqrt(mean(x^2) + eps)) * g. One wavefront per row,
// four rows per 256-thread block; the row stays in registers (d <= 64 * kMaxPer).

constexpr int kMaxPer = 24;   // d <= 1536

// Every global load of these kernels is unconditional (lanes past d re-read
// entry d - 1 and zero it afterwards): a load inside a guarded block makes the
// compiler wait for each load before the next one.
template <int PER>
__device__ inline void load_gain(const float* __restrict__ g, int d, float (&gv)[PER]) {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int k = 0; k < PER; ++k) gv[k] = g[min(lane + 64 * k, d - 1)];
}

template <typename T, int PER>
__device__ inline void norm_store(const float (&x)[PER], const float (&gv)[PER], float eps, int d,
                                  T* __restrict__ out) {
    const int lane = threadIdx.x & 63;
    float ss = 0.f;
#pragma unroll
    for (int k = 0; k < PER; ++k) ss = fmaf(x[k], x[k], ss);
    ss = wave_sum(ss);
    const float r = 1.0f / sqrtf(ss / (float)d + eps);
#pragma unroll
    for (int k = 0; k < PER; ++k) {
        const int i = lane + 64 * k;
        if (i < d) Elem<T>::store(out + i, (x[k] * r) * gv[k]);
    }
}

template <typename T, int PER>
__global__ __launch_bounds__(256) void k_embed_norm(RowMeta rows, const int* nrows_dev, int cap,
                                                    const float* __restrict__ tok_emb,
                                                    const float* __restrict__ cls_emb,
                                                    const float* __restrict__ g, float eps, int d,
                                                    float* __restrict__ h, T* __restrict__ hb) {
    const int r = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
    if (r >= cap) return;
    // the gain, the row count and the token are fetched together (tok[r] is
    // allocated for every r below the capacity); only the gather waits
    float gv[PER];
    load_gain(g, d, gv);
    const int nrows = *nrows_dev;
    const int tok = rows.tok[r];
    if (r >= nrows) return;
    const float* e = tok >= 0 ? tok_emb + (size_t)tok * d : cls_emb + (size_t)(-(tok + 1)) * d;
    float x[PER];
#pragma unroll
    for (int k = 0; k < PER; ++k) x[k] = e[min(lane + 64 * k, d - 1)];
#pragma unroll
    for (int k = 0; k < PER; ++k)
        if (lane + 64 * k >= d) x[k] = 0.f;
#pragma unroll
    for (int k = 0; k < PER; ++k) {
        const int i = lane + 64 * k;
        if (i < d) h[(size_t)r * d + i] = x[k];
    }
    norm_store<T, PER>(x, gv, eps, d, hb + (size_t)r * d);
}

template <typename T, int PER>
__global__ __launch_bounds__(256) void k_rmsnorm(const float* __restrict__ h,
                                                 const int32_t* src_idx, const int* nrows_dev,
                                                 int cap, const float* __restrict__ g, float eps,
                                                 int d, T* __restrict__ hb) {
    const int r = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
    if (r >= cap) return;
    float gv[PER];
    load_gain(g, d, gv);
    const int nrows = *nrows_dev;
    const int src = src_idx ? src_idx[r] : r;   // fetched with the count (r is below the capacity)
    if (r >= nrows) return;
    float x[PER];
#pragma unroll
    for (int k = 0; k < PER; ++k) x[k] = h[(size_t)src * d + min(lane + 64 * k, d - 1)];
#pragma unroll
    for (int k = 0; k < PER; ++k)
        if (lane + 64 * k >= d) x[k] = 0.f;
    norm_store<T, PER>(x, gv, eps, d, hb + (size_t)r * d);
}

// the per-lane element count of a row of d (a multiple of 64 in fp16 mode)
template <typename F>
static void by_per(int d, F f) {
    const int per = (d + 63) / 64;
    if (per <= 1) f(std::integral_constant<int, 1>{});
    else if (per <= 4) f(std::integral_constant<int, 4>{});
    else if (per <= 12) f(std::integral_constant<int, 12>{});
    else if (per <= 16) f(std::integral_constant<int, 16>{});
    else if (per <= 20) f(std::integral_constant<int, 20>{});
    else f(std::integral_constant<int, 24>{});
}

void embed_norm(bool f16, const RowMeta& rows, const int* nrows_dev, int nrows_cap,
                const float* tok_emb, const float* cls_emb, const float* gain, float eps, int d,
                float* h, void* hb, hipStream_t s) {
    if (nrows_cap <= 0) return;
    const dim3 grid((nrows_cap + 3) / 4);
    by_per(d, [&](auto P) {
        constexpr int PER = decltype(P)::value;
        if (f16)
            launch(k_embed_norm<uint16_t, PER>, grid, dim3(256), 0, s, rows, nrows_dev, nrows_cap,
                   tok_emb, cls_emb, gain, eps, d, h, (uint16_t*)hb);
        else
            launch(k_embed_norm<float, PER>, grid, dim3(256), 0, s, rows, nrows_dev, nrows_cap,
                   tok_emb, cls_emb, gain, eps, d, h, (float*)hb);
    });
}

void rmsnorm(bool f16, const float* h, const int32_t* src_idx, const int* nrows_dev,
             int nrows_cap, const float* gain, float eps, int d, void* hb, hipStream_t s) {
    if (nrows_cap <= 0) return;
    const dim3 grid((nrows_cap + 3) / 4);
    by_per(d, [&](auto P) {
        constexpr int PER = decltype(P)::value;
        if (f16)
            launch(k_rmsnorm<uint16_t, PER>, grid, dim3(256), 0, s, h, src_idx, nrows_dev,
                   nrows_cap, gain, eps, d, (uint16_t*)hb);
        else
            launch(k_rmsnorm<float, PER>, grid, dim3(256), 0, s, h, src_idx, nrows_dev,
                   nrows_cap, gain, eps, d, (float*)hb);
    });
}

// One 64-lane block per row. Lane l holds dims 4 l + 256 k .. + 3 for k < NV4,
// read as float4 (d is a multiple of 4; chunks past d are clamped on load and
// never stored).
template <typename T, int NV4>
__global__ __launch_bounds__(64) void k_reduce_norm(const float* __restrict__ part, int splits,
                                                    int m_cap, float* __restrict__ h,
                                                    const int* nrows_dev,
                                                    const float* __restrict__ g, float eps, int d,
                                                    T* __restrict__ hb) {
    constexpr int kSplitMax = 4;
    const int r = blockIdx.x, lane = threadIdx.x;
    if (r >= m_cap) return;
    // the row count first: the grid covers the capacity, and rows at or past
    // the count (most of them in the last rounds) load and store nothing.
    // Then one phase of loads: every split's partial (splits = 0: the
    // projection has already added its sum into h), the residual and the gain.
    const int nrows = *nrows_dev;
    if (r >= nrows) return;
    const int nv = d >> 2;
    float4 pz[kSplitMax][NV4], hv[NV4], gv[NV4];
#pragma unroll
    for (int k = 0; k < NV4; ++k) {
        const int c = min(lane + 64 * k, nv - 1);
        if (splits > 0) {
#pragma unroll
            for (int z = 0; z < kSplitMax; ++z) {
                const int zz = min(z, splits - 1);
                pz[z][k] = reinterpret_cast<const float4*>(part + ((size_t)zz * m_cap + r) * d)[c];
            }
        }
        hv[k] = reinterpret_cast<const float4*>(h + (size_t)r * d)[c];
        gv[k] = reinterpret_cast<const float4*>(g)[c];
    }
    float4 x[NV4];
    float ss = 0.f;
#pragma unroll
    for (int k = 0; k < NV4; ++k) {
        const bool in = lane + 64 * k < nv;
        if (splits > 0) {
            float4 acc = pz[0][k];
#pragma unroll
            for (int z = 1; z < kSplitMax; ++z)
                if (z < splits) {   // split order
                    acc.x += pz[z][k].x;
                    acc.y += pz[z][k].y;
                    acc.z += pz[z][k].z;
                    acc.w += pz[z][k].w;
                }
            x[k] = make_float4(hv[k].x + acc.x, hv[k].y + acc.y, hv[k].z + acc.z, hv[k].w + acc.w);
        } else {
            x[k] = hv[k];
        }
        if (in) {
            ss = fmaf(x[k].x, x[k].x, ss);
            ss = fmaf(x[k].y, x[k].y, ss);
            ss = fmaf(x[k].z, x[k].z, ss);
            ss = fmaf(x[k].w, x[k].w, ss);
        }
    }
    if (splits > 0) {
#pragma unroll
        for (int k = 0; k < NV4; ++k)
            if (lane + 64 * k < nv) reinterpret_cast<float4*>(h + (size_t)r * d)[lane + 64 * k] = x[k];
    }
    if (!hb) return;
    ss = wave_sum(ss);
    const float rn = 1.0f / sqrtf(ss / (float)d + eps);
#pragma unroll
    for (int k = 0; k < NV4; ++k) {
        const int i = 4 * (lane + 64 * k);
        if (i < d) {
            Elem<T>::store(hb + (size_t)r * d + i + 0, (x[k].x * rn) * gv[k].x);
            Elem<T>::store(hb + (size_t)r * d + i + 1, (x[k].y * rn) * gv[k].y);
            Elem<T>::store(hb + (size_t)r * d + i + 2, (x[k].z * rn) * gv[k].z);
            Elem<T>::store(hb + (size_t)r * d + i + 3, (x[k].w * rn) * gv[k].w);
        }
    }
}

template <typename T, int NV4>
static void reduce_norm_launch(const float* part, int splits, int m_cap, float* h,
                               const int* nrows_dev, const float* gain, float eps, int d, void* hb,
                               hipStream_t s) {
    launch(k_reduce_norm<T, NV4>, dim3(m_cap), dim3(64), 0, s, part, splits, m_cap, h,
           nrows_dev, gain, eps, d, (T*)hb);
}

template <typename T>
static void reduce_norm_dispatch(const float* part, int splits, int m_cap, float* h,
                                 const int* nrows_dev, const float* gain, float eps, int d,
                                 void* hb, hipStream_t s) {
    switch ((d + 255) / 256) {
        case 1: reduce_norm_launch<T, 1>(part, splits, m_cap, h, nrows_dev, gain, eps, d, hb, s); break;
        case 2: reduce_norm_launch<T, 2>(part, splits, m_cap, h, nrows_dev, gain, eps, d, hb, s); break;
        case 3: reduce_norm_launch<T, 3>(part, splits, m_cap, h, nrows_dev, gain, eps, d, hb, s); break;
        case 4: reduce_norm_launch<T, 4>(part, splits, m_cap, h, nrows_dev, gain, eps, d, hb, s); break;
        case 5: reduce_norm_launch<T, 5>(part, splits, m_cap, h, nrows_dev, gain, eps, d, hb, s); break;
        default: reduce_norm_launch<T, 6>(part, splits, m_cap, h, nrows_dev, gain, eps, d, hb, s); break;
    }
}

void reduce_residual_norm(bool f16, const float* part, int splits, int m_cap, float* h,
                          const int* nrows_dev, const float* gain, float eps, int d, void* hb,
                          hipStream_t s) {
    if (m_cap <= 0) return;
    if (f16)
        reduce_norm_dispatch<uint16_t>(part, splits, m_cap, h, nrows_dev, gain, eps, d, hb, s);
    else
        reduce_norm_dispatch<float>(part, splits, m_cap, h, nrows_dev, gain, eps, d, hb, s);
}

// ---------------------------------------------------------------- Philox test entry
__global__ void k_philox(uint64_t seed, int n, const uint32_t* bt, uint32_t* out) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    const U4 r = philox4x32_10(seed, bt[2 * i], bt[2 * i + 1], 0u, 0u);
    out[4 * i + 0] = r.x;
    out[4 * i + 1] = r.y;
    out[4 * i + 2] = r.z;
    out[4 * i + 3] = r.w;
}

void philox_fill(uint64_t seed, int n, const uint32_t* bt, uint32_t* out, hipStream_t s) {
    if (n <= 0) return;
    launch(k_philox, dim3((n + 255) / 256), dim3(256), 0, s, seed, n, bt, out);
}

}  // namespace hbsjd
