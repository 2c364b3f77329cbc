// Sampling side of a round: the distribution transform of every verifier row,
// probabilistic (Sec. 4.2, Eq. 5) or greedy (Eq. 4) verification of each
// image's window, commit, and the Jacobi window refresh (reused predictions
// first, history tokens at offset H for the rest; Sec. 4.2).
//
// Every fp32 sum over the vocabulary is associated the same way: sequential
// inside consecutive 64-entry chunks, then the chunk totals sequential. The
// inverse CDF returns the first entry whose prefix (chunk prefix plus in-chunk
// prefix) exceeds u * total. Contraction is off in this file so each operation
// rounds once.
#include "common.h"
#include "launch.h"

#pragma clang fp contract(off)

namespace hbsjd {

constexpr int kBins = 1024;     // histogram bins of the top-k threshold search
constexpr int kCand = 256;      // candidates ranked exactly once the bin is this small

// ---------------------------------------------------------------- row staging
// A 256-thread block holds one vocabulary row with thread t owning chunk t
// (entries [64 t, 64 t + 64)) in registers: the layout every pinned chunk sum
// needs. Global memory is read and written in whole 1 KB wavefront accesses and
// transposed through LDS, half of a wavefront's chunks at a time: in half h,
// stage[w][j] holds chunk 64 w + 32 h + j, padded to 68 floats so the owners'
// 16-byte reads fall in distinct banks. Every thread of the block must call.
constexpr int kStageStride = kChunk + 4;
constexpr int kStageFloats = 4 * 32 * kStageStride;   // 34,816 bytes

// op(k, x) receives entry 64 t + k of the calling thread for k = 0..63 (0 past
// V; V is a multiple of 4)
template <typename Op>
__device__ __forceinline__ void stage_load_row(const float* __restrict__ row, int V, float* stage,
                                               Op op) {
    const int t = threadIdx.x, lane = t & 63, w = t >> 6;
    float* sw = stage + w * 32 * kStageStride;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const int base = (64 * w + 32 * h) * kChunk;
        float4 x[8];
        // unconditional loads (entries past V re-read the row's last float4)
        // so all eight stay in flight together; the zeroing past V is a
        // select taken once they have landed (overwriting a register whose
        // load is still in flight would make the compiler wait for it)
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int v = base + 256 * i + 4 * lane;
            x[i] = *reinterpret_cast<const float4*>(row + (v < V ? v : V - 4));
        }
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int e = 256 * i + 4 * lane;
            const bool in = base + e < V;
            const float4 y = make_float4(in ? x[i].x : 0.f, in ? x[i].y : 0.f, in ? x[i].z : 0.f,
                                         in ? x[i].w : 0.f);
            *reinterpret_cast<float4*>(sw + (e >> 6) * kStageStride + (e & 63)) = y;
        }
        __syncthreads();
        if ((lane >> 5) == h) {
            const float* mine = sw + (lane & 31) * kStageStride;
#pragma unroll
            for (int k = 0; k < kChunk; k += 4) {
                const float4 y = *reinterpret_cast<const float4*>(mine + k);
                op(k, y.x);
                op(k + 1, y.y);
                op(k + 2, y.z);
                op(k + 3, y.w);
            }
        }
        __syncthreads();
    }
}

// writes row[0, V): val(k) gives entry 64 t + k of the calling thread
template <typename Val>
__device__ __forceinline__ void stage_store_row(float* __restrict__ row, int V, float* stage,
                                                Val val) {
    const int t = threadIdx.x, lane = t & 63, w = t >> 6;
    float* sw = stage + w * 32 * kStageStride;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const int base = (64 * w + 32 * h) * kChunk;
        if ((lane >> 5) == h) {
            float* mine = sw + (lane & 31) * kStageStride;
#pragma unroll
            for (int k = 0; k < kChunk; k += 4)
                *reinterpret_cast<float4*>(mine + k) = make_float4(val(k), val(k + 1), val(k + 2), val(k + 3));
        }
        __syncthreads();
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int e = 256 * i + 4 * lane;
            const int v = base + e;
            const float4 x = *reinterpret_cast<const float4*>(sw + (e >> 6) * kStageStride + (e & 63));
            if (v < V) *reinterpret_cast<float4*>(row + v) = x;
        }
        __syncthreads();
    }
}

// One thread's sequential sums over LDS in the pinned order. The reads of
// each group of 16 entries are issued before the adds of the previous group,
// so the chain of adds does not wait on an LDS round trip every few entries.
// seq_sum_lds returns ((v[0] + v[1]) + ...) + v[n-1] (0 + ... from zero);
// seq_prefix_lds turns v[0..n-1] into its inclusive running sums from zero.
constexpr int kSeqGroup = 16;
__device__ inline float seq_sum_lds(const float* v, int n) {
    float z = 0.f;
    const int groups = n / kSeqGroup;
    if (groups > 0) {
        float cur[kSeqGroup];
#pragma unroll
        for (int k = 0; k < kSeqGroup; ++k) cur[k] = v[k];
        for (int g = 1; g < groups; ++g) {
            float nxt[kSeqGroup];
#pragma unroll
            for (int k = 0; k < kSeqGroup; ++k) nxt[k] = v[kSeqGroup * g + k];
#pragma unroll
            for (int k = 0; k < kSeqGroup; ++k) z = z + cur[k];
#pragma unroll
            for (int k = 0; k < kSeqGroup; ++k) cur[k] = nxt[k];
        }
#pragma unroll
        for (int k = 0; k < kSeqGroup; ++k) z = z + cur[k];
    }
    for (int i = kSeqGroup * groups; i < n; ++i) z = z + v[i];
    return z;
}
__device__ inline void seq_prefix_lds(float* v, int n) {
    float run = 0.f;
    const int groups = n / kSeqGroup;
    if (groups > 0) {
        float cur[kSeqGroup];
#pragma unroll
        for (int k = 0; k < kSeqGroup; ++k) cur[k] = v[k];
        for (int g = 1; g < groups; ++g) {
            float nxt[kSeqGroup];
#pragma unroll
            for (int k = 0; k < kSeqGroup; ++k) nxt[k] = v[kSeqGroup * g + k];
#pragma unroll
            for (int k = 0; k < kSeqGroup; ++k) {
                run = run + cur[k];
                v[kSeqGroup * (g - 1) + k] = run;
            }
#pragma unroll
            for (int k = 0; k < kSeqGroup; ++k) cur[k] = nxt[k];
        }
#pragma unroll
        for (int k = 0; k < kSeqGroup; ++k) {
            run = run + cur[k];
            v[kSeqGroup * (groups - 1) + k] = run;
        }
    }
    for (int i = kSeqGroup * groups; i < n; ++i) {
        run = run + v[i];
        v[i] = run;
    }
}

// order-preserving map of a float to an int (and back), for exact LDS min/max
__device__ inline int float_key(float f) {
    const int i = __builtin_bit_cast(int, f);
    return i >= 0 ? i : i ^ 0x7fffffff;
}
__device__ inline float key_float(int k) {
    return __builtin_bit_cast(float, k >= 0 ? k : k ^ 0x7fffffff);
}

// ---------------------------------------------------------------- transform
// One 256-thread block per distribution row; thread c owns vocabulary chunk c
// (64 consecutive entries) in registers.
__global__ __launch_bounds__(256) void k_transform(TransformArgs a) {
    __shared__ float red[4];
    __shared__ int ired[8];
    __shared__ int hist[kBins];
    __shared__ float tot[kMaxChunks + 1];
    __shared__ float cand[kCand];
    __shared__ int s_int[4];
    __shared__ int s_mm[2];
    __shared__ float s_flt[4];
    __shared__ __attribute__((aligned(16))) float stage[kStageFloats];

    const int r = blockIdx.x;
    if (r >= min(*a.nout_dev, a.nout_cap)) return;
    const int t = threadIdx.x;
    const int V = a.V;
    const int nC = (V + kChunk - 1) / kChunk;
    const int s = r / a.rows_per_slot, i = r - s * a.rows_per_slot;
    const int b = a.slot_img[s];
    const float tau = a.temperature[b];
    // the draw below needs the image's cursor and the seed: fetched now, with
    // the row, rather than after the reductions
    const int pos = min(a.cursor[b], a.T) + i + 1;
    const float u_draft = uniforms_at(meta_seed(a.meta), b, pos).draft;
    const float* lc = a.logits + (size_t)((s * a.cfg) * a.rows_per_slot + i) * V;
    const float* lu = a.cfg == 2 ? a.logits + (size_t)((s * 2 + 1) * a.rows_per_slot + i) * V : nullptr;

    // guided logits, temperature, max and argmax (of the guided logits)
    float y[kChunk];
    stage_load_row(lc, V, stage, [&](int k, float x) { y[k] = x; });
    if (lu) stage_load_row(lu, V, stage, [&](int k, float x) { y[k] = x + a.cfg_scale * (y[k] - x); });
    float lmax = -INFINITY, ymax = -INFINITY, ymin = INFINITY;
    int lidx = 0x7fffffff;
    int nan_seen = 0;
    const int v0 = t * kChunk;
#pragma unroll
    for (int k = 0; k < kChunk; ++k) {
        const int v = v0 + k;
        const float l = y[k];
        const float yy = l / tau;
        // entries past V become NaN, which every range test and the softmax's
        // threshold test below reject
        y[k] = v < V ? yy : __builtin_nanf("");
        if (v < V) {
            if (l != l) nan_seen = 1;
            if (l > lmax) { lmax = l; lidx = v; }
            ymax = fmaxf(ymax, yy);
            ymin = fminf(ymin, yy);
        }
    }
    if (nan_seen) atomicOr(&a.meta[kMetaError], (int)kErrNanLogit);
    // argmax with the lowest index on ties
    {
        float m = lmax;
        int idx = lidx;
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) {
            const float m2 = __shfl_xor(m, o, 64);
            const int i2 = __shfl_xor(idx, o, 64);
            if (m2 > m || (m2 == m && i2 < idx)) { m = m2; idx = i2; }
        }
        if ((t & 63) == 0) { red[t >> 6] = m; ired[t >> 6] = idx; }
        __syncthreads();
        if (t == 0) {
            float bm = red[0];
            int bi = ired[0];
            for (int w = 1; w < 4; ++w)
                if (red[w] > bm || (red[w] == bm && ired[w] < bi)) { bm = red[w]; bi = ired[w]; }
            a.amax[r] = bi;
        }
        __syncthreads();
    }
    ymax = block_reduce(ymax, red, [](float p, float q) { return fmaxf(p, q); });

    // top-k threshold: the k-th largest y counting ties (exact)
    float thr = -INFINITY;
    if (a.top_k > 0 && a.top_k < V) {
        ymin = block_reduce(ymin, red, [](float p, float q) { return fminf(p, q); });
        float lo = ymin, hi = ymax;
        int above = 0;   // entries strictly above the current range
        for (int iter = 0; iter < 64; ++iter) {
            if (lo == hi) { thr = lo; break; }
            for (int k = t; k < kBins; k += 256) hist[k] = 0;
            __syncthreads();
            const float scale = (float)kBins / (hi - lo);
            // each pass over the entries takes its own copies of the range,
            // which the compiler cannot see through: otherwise it keeps the 64
            // range tests of one pass alive for the next ones (128 SGPRs,
            // spilled to VGPRs)
            float lo_h = lo, hi_h = hi, scale_h = scale;
            asm volatile("" : "+v"(lo_h), "+v"(hi_h), "+v"(scale_h));
#pragma unroll
            for (int k = 0; k < kChunk; ++k) {
                const float yy = y[k];
                if (yy >= lo_h && yy <= hi_h) {
                    int bin = (int)((yy - lo_h) * scale_h);
                    bin = bin > kBins - 1 ? kBins - 1 : bin;
                    atomicAdd(&hist[bin], 1);
                }
            }
            __syncthreads();
            // suffix counts: thread t owns bins 4t..4t+3
            int own = 0;
#pragma unroll
            for (int q = 0; q < 4; ++q) own += hist[4 * t + q];
            // inclusive suffix scan over threads (higher threads = higher bins)
            int sfx = own;
            {
                const int lane = t & 63, wv = t >> 6;
#pragma unroll
                for (int o = 1; o < 64; o <<= 1) {
                    const int yv = __shfl_down(sfx, o, 64);
                    if (lane + o < 64) sfx += yv;
                }
                if (lane == 0) ired[wv] = sfx;
                __syncthreads();
                for (int w = wv + 1; w < 4; ++w) sfx += ired[w];
                __syncthreads();
            }
            // entries in bins above thread t's group
            int cum = above + sfx - own;
            if (t == 0) {
                s_int[0] = -1;
                s_int[1] = 0;
                s_int[2] = 0;
                s_mm[0] = 0x7fffffff;
                s_mm[1] = (int)0x80000000;
            }
            __syncthreads();
            for (int q = 3; q >= 0; --q) {
                const int hb = hist[4 * t + q];
                if (cum < a.top_k && a.top_k <= cum + hb) {
                    s_int[0] = 4 * t + q;
                    s_int[1] = cum;
                    s_int[2] = hb;
                }
                cum += hb;
            }
            __syncthreads();
            const int bstar = s_int[0];
            const int above_new = s_int[1];
            const int cnt = s_int[2];
            __syncthreads();
            if (bstar < 0) {   // only with NaN logits, which are reported as an error
                thr = lo;
                break;
            }
            // the bins are recomputed below with the same arithmetic from copies
            // the compiler cannot see through, so it does not keep all 64 of
            // this thread's bins alive across the scan
            float lo_b = lo, scale_b = scale;
            asm volatile("" : "+v"(lo_b), "+v"(scale_b));
            if (cnt <= kCand) {
                if (t == 0) s_int[3] = 0;
                __syncthreads();
                float lo_c = lo, hi_c = hi;
                asm volatile("" : "+v"(lo_c), "+v"(hi_c));
#pragma unroll
                for (int k = 0; k < kChunk; ++k) {
                    const float yy = y[k];
                    if (yy >= lo_c && yy <= hi_c) {
                        int bin = (int)((yy - lo_b) * scale_b);
                        bin = bin > kBins - 1 ? kBins - 1 : bin;
                        if (bin == bstar) cand[atomicAdd(&s_int[3], 1)] = yy;
                    }
                }
                __syncthreads();
                const int need = a.top_k - above_new;   // rank inside the bin, 1-based
                if (t < cnt) {
                    const float cv = cand[t];
                    int gt = 0, ge = 0;
                    for (int j = 0; j < cnt; ++j) {
                        gt += cand[j] > cv;
                        ge += cand[j] >= cv;
                    }
                    if (gt < need && need <= ge) s_flt[0] = cv;
                }
                __syncthreads();
                thr = s_flt[0];
                break;
            }
            // narrow to the values that fell into the chosen bin: their exact
            // minimum and maximum, on an order-preserving integer image of the
            // float: per thread (chains cut every 8 entries, so the compiler
            // does not rebalance them into trees), per wavefront, then across
            // the block through LDS atomics. The images are formed from a
            // copy of the entries the compiler cannot see through, so it does
            // not hoist all 64 of them out of the search loop
            {
                float lo_n = lo, hi_n = hi;
                int zero = 0;
                asm volatile("" : "+v"(lo_n), "+v"(hi_n), "+v"(zero));
                int mn = 0x7fffffff, mx = (int)0x80000000;
#pragma unroll
                for (int k = 0; k < kChunk; ++k) {
                    if ((k & 7) == 0) asm volatile("" : "+v"(mn), "+v"(mx));
                    const float yy = y[k];
                    int bin = (int)((yy - lo_b) * scale_b);
                    bin = bin > kBins - 1 ? kBins - 1 : bin;
                    const bool sel = yy >= lo_n && yy <= hi_n && bin == bstar;
                    const int bits = __float_as_int(yy) | zero;
                    const int key = bits >= 0 ? bits : bits ^ 0x7fffffff;
                    mn = sel && key < mn ? key : mn;
                    mx = sel && key > mx ? key : mx;
                }
                mn = wave_min_int(mn);
                mx = wave_max_int(mx);
                if ((t & 63) == 0) {
                    atomicMin(&s_mm[0], mn);
                    atomicMax(&s_mm[1], mx);
                }
            }
            __syncthreads();
            lo = key_float(s_mm[0]);
            hi = key_float(s_mm[1]);
            __syncthreads();
            above = above_new;
            thr = lo;   // only reached if the loop runs out: keeps at least k entries
        }
    }

    // softmax over the kept entries; Z in the pinned chunk order
    float csum = 0.f;
#pragma unroll
    for (int k = 0; k < kChunk; ++k) {
        const float e = (y[k] >= thr) ? expf(y[k] - ymax) : 0.f;
        y[k] = e;
        csum = csum + e;
    }
    if (t < nC) tot[t] = csum;
    __syncthreads();
    if (t == 0) {
        s_flt[1] = seq_sum_lds(tot, nC);
        s_int[2] = -1;   // the row's last positive entry, gathered below
    }
    __syncthreads();
    const float z = s_flt[1];
    float* prow = a.p + (size_t)r * V;
    float psum = 0.f;
    uint64_t pos_mask = 0;   // entries past V are 0, so never positive
#pragma unroll
    for (int k = 0; k < kChunk; ++k) {
        y[k] = y[k] / z;
        psum = psum + y[k];
        pos_mask |= (uint64_t)(y[k] > 0.f) << k;
    }
    // this thread's last positive entry (the fallback of the draw below)
    const int last_pos = pos_mask ? v0 + 63 - __clzll((long long)pos_mask) : -1;
    stage_store_row(prow, V, stage, [&](int k) { return y[k]; });
    // chunk prefix of p: tot[c] becomes the sum of chunks 0..c-1 (pinned order)
    if (t < nC) tot[t + 1] = psum;
    {
        const int lw = wave_max_int(last_pos);
        if ((t & 63) == 0) atomicMax(&s_int[2], lw);
    }
    __syncthreads();
    if (t == 0) {
        tot[0] = 0.f;
        seq_prefix_lds(tot + 1, nC);
    }
    __syncthreads();

    // draft candidate of this row: the position it predicts is n_b + i + 1 no
    // matter how the round's verification ends, so its draw from p with
    // u_draft(b, n_b + i + 1) is taken here, with the row's own prefix: the
    // same sums and search as block_inv_cdf_regs over the stored row, hence
    // the same token
    int z_draft = -1;
    if (pos <= a.T) {
        const float target = u_draft * tot[nC];
        if (t < 64) {
            int cs = 0x7fffffff;
            for (int c = t; c < nC; c += 64)
                if (tot[c + 1] > target) { cs = c; break; }
            cs = wave_min_int(cs);
            if (t == 0) s_int[0] = cs;
        }
        __syncthreads();
        const int cs = s_int[0];
        if (cs == 0x7fffffff) {   // rounding left the target above the total
            z_draft = s_int[2];
        } else {
            // the owner parks its chunk in LDS and thread 0 scans it in order
            if (t == cs) {
#pragma unroll
                for (int k = 0; k < kChunk; k += 4)
                    *reinterpret_cast<float4*>(&cand[k]) = make_float4(y[k], y[k + 1], y[k + 2], y[k + 3]);
            }
            __syncthreads();
            if (t == 0) {   // the chunk's entries in order; LDS loads issued ahead of the adds
                const float before = tot[cs];
                const int nk = min(kChunk, V - cs * kChunk);
                float xb[kChunk];
#pragma unroll
                for (int k = 0; k < kChunk; k += 4) {
                    const float4 q4 = *reinterpret_cast<const float4*>(&cand[k]);
                    xb[k] = q4.x;
                    xb[k + 1] = q4.y;
                    xb[k + 2] = q4.z;
                    xb[k + 3] = q4.w;
                }
                float inner = 0.f;
                int found = -1, lastpos = -1;
#pragma unroll
                for (int k = 0; k < kChunk; ++k)
                    if (found < 0 && k < nk) {
                        inner = inner + xb[k];
                        if (xb[k] > 0.f) lastpos = cs * kChunk + k;
                        if (before + inner > target) found = cs * kChunk + k;
                    }
                s_int[1] = found >= 0 ? found : lastpos;
            }
            __syncthreads();
            z_draft = s_int[1];
        }
    }
    if (t == 0) a.samp[r] = z_draft;
}

void transform(const TransformArgs& a, hipStream_t s) {
    if (a.nout_cap <= 0) return;
    launch(k_transform, dim3(a.nout_cap), dim3(256), 0, s, a);
}

// ---------------------------------------------------------------- inverse CDF helpers

// Block-level inverse CDF over non-negative weights held chunk-owned in
// registers (thread t has entries 64 t .. 64 t + 63 in w), in the pinned
// association: the first entry whose chunk prefix plus in-chunk prefix exceeds
// u * total, else the last positive entry. Returns -1 when every weight is
// zero. All 256 threads must call it.
__device__ inline int block_inv_cdf_regs(const float (&w)[kChunk], int V, float u, float* cp,
                                         int* res) {
    const int t = threadIdx.x;
    const int nC = (V + kChunk - 1) / kChunk;
    const int v0 = t * kChunk;
    float sum = 0.f;
    int last = -1;
#pragma unroll
    for (int k = 0; k < kChunk; ++k)
        if (v0 + k < V) {
            sum = sum + w[k];
            if (w[k] > 0.f) last = v0 + k;
        }
    if (t < nC) cp[t + 1] = sum;
    __syncthreads();
    if (t == 0) {
        cp[0] = 0.f;
        seq_prefix_lds(cp + 1, nC);
    }
    __syncthreads();
    const float total = cp[nC];
    if (!(total > 0.f)) return -1;
    const float target = u * total;
    if (t < 64) {
        int cs = 0x7fffffff;
        for (int c = t; c < nC; c += 64)
            if (cp[c + 1] > target) { cs = c; break; }
        cs = wave_min_int(cs);
        if (t == 0) *res = cs;
    }
    __syncthreads();
    const int cs = *res;
    __syncthreads();
    if (cs == 0x7fffffff) {   // rounding left the target above the total: last positive entry
        const int lw = wave_max_int(last);
        if (t == 0) *res = -1;
        __syncthreads();
        if ((t & 63) == 0) atomicMax(res, lw);
    } else if (t == cs) {
        const float before = cp[cs];
        float inner = 0.f;
        int found = -1, lastpos = -1;
#pragma unroll
        for (int k = 0; k < kChunk; ++k) {
            if (found < 0 && v0 + k < V) {
                inner = inner + w[k];
                if (w[k] > 0.f) lastpos = v0 + k;
                if (before + inner > target) found = v0 + k;
            }
        }
        *res = found >= 0 ? found : lastpos;
    }
    __syncthreads();
    return *res;
}

// The replacement token of a rejected draft (Sec. 4.2, Eq. 5): a draw with u
// from the residual max(0, p - q), where q is the proposal row `qrow`, or a
// point mass on z when qrow is null (a history draft); from p itself when the
// residual is zero everywhere in fp32. All 256 threads must call it.
__device__ __forceinline__ int replacement_draw(const float* __restrict__ pr,
                                                const float* __restrict__ qrow, int z, int V,
                                                float u, float* stage, float* cp, int* res) {
    const int t = threadIdx.x;
    float w[kChunk];
    stage_load_row(pr, V, stage, [&](int k, float x) { w[k] = x; });
    if (qrow) {
        stage_load_row(qrow, V, stage, [&](int k, float x) {
            const float d = w[k] - x;
            w[k] = d > 0.f ? d : 0.f;
        });
    } else {
#pragma unroll
        for (int k = 0; k < kChunk; ++k) {
            const float d = w[k] - (t * kChunk + k == z ? 1.0f : 0.0f);
            w[k] = d > 0.f ? d : 0.f;
        }
    }
    int rep = block_inv_cdf_regs(w, V, u, cp, res);
    if (rep < 0) {   // the residual underflowed: draw from p
        stage_load_row(pr, V, stage, [&](int k, float x) { w[k] = x; });
        rep = block_inv_cdf_regs(w, V, u, cp, res);
    }
    return rep;
}

// ---------------------------------------------------------------- verify + commit + refresh
// One 256-thread block per processed image.
__global__ __launch_bounds__(256) void k_verify(VerifyArgs a) {
    __shared__ float cp[kMaxChunks + 1];
    __shared__ __attribute__((aligned(16))) float stage[kStageFloats];
    __shared__ int s_res;
    __shared__ int s_first;
    __shared__ int old_dr[64], old_q[64];
    __shared__ int new_dr[64], new_q[64];

    const int sl = blockIdx.x;
    if (sl >= min(*a.nimg_dev, a.nimg_cap)) return;
    const int t = threadIdx.x;
    const int b = a.slot_img[sl];
    const int n = a.cursor[b];
    if (n >= a.T) return;              // finished image in Full mode: rows discarded
    const int W = a.W, V = a.V, R = a.rows_per_slot;
    const uint64_t seed = meta_seed(a.meta);
    if (a.ar) {
        // cached AR: the image's single row predicts position n + 1 (Eq. 1)
        if (t >= 64) return;
        const int prow = sl * R;
        const int z = a.greedy ? a.amax[prow] : a.samp[prow];
        if (t == 0) {
            a.xtok[(size_t)b * a.T + n] = z;
            const int round = a.meta[kMetaRound];
            if (a.counts && round >= 0 && round < a.max_rounds) a.counts[(size_t)round * a.B + b] = 1;
            atomicAdd((unsigned long long*)&a.stats[0], 1ull);
            atomicAdd((unsigned long long*)&a.stats[2], 1ull);
            a.cursor[b] = n + 1;
        }
        return;
    }
    int n_new, base, nrows;
    if (a.prefill) {
        n_new = n;
        base = n;
        nrows = 1;
    } else {
        // the batch-synchronous ablation stops at the image's window end; an
        // image already there verifies nothing and only re-draws its window
        const int We = max(min(W, (a.win_end ? a.win_end[b] : a.T) - n), 0);
        if (t < W) {
            old_dr[t] = a.drafts[(size_t)b * W + t];
            old_q[t] = a.qsrc[(size_t)b * W + t];
        }
        if (t == 0) s_first = We + 1;
        __syncthreads();
        if (t < We) {
            const int j = t + 1;
            const int z = old_dr[t];
            const int prow = sl * R + (j - 1);
            bool acc;
            if (a.greedy) {
                acc = z == a.amax[prow];
            } else {
                const float P = a.p[(size_t)prow * V + z];
                const int qs = old_q[t];
                const float Q = qs >= 0 ? a.p_prev[(size_t)qs * V + z] : 1.0f;
                if (!(Q > 0.f)) atomicOr(&a.meta[kMetaError], (int)kErrZeroProposal);
                const float u = uniforms_at(seed, b, n + j).acc;
                acc = (P >= Q) || (u < P / Q);
            }
            if (!acc) atomicMin(&s_first, j);
        }
        __syncthreads();
        const int js = s_first;
        const bool rejected = js <= We;
        const int count = rejected ? js : We;
        int rep = 0;
        if (rejected) {
            const int prow = sl * R + (js - 1);
            if (a.greedy) {
                rep = a.amax[prow];
            } else {
                const int qs = old_q[js - 1];
                const float u = uniforms_at(seed, b, n + js).res;
                rep = replacement_draw(a.p + (size_t)prow * V,
                                       qs >= 0 ? a.p_prev + (size_t)qs * V : nullptr,
                                       old_dr[js - 1], V, u, stage, cp, &s_res);
            }
        }
        // commit x_{n+1..n+count}
        if (t < count) {
            const int tok = (t == count - 1 && rejected) ? rep : old_dr[t];
            a.xtok[(size_t)b * a.T + n + t] = tok;
        }
        if (t == 0) {
            const int round = a.meta[kMetaRound];
            if (a.counts && round >= 0 && round < a.max_rounds) a.counts[(size_t)round * a.B + b] = count;
            atomicAdd((unsigned long long*)&a.stats[0], (unsigned long long)count);
            atomicAdd((unsigned long long*)&a.stats[1], (unsigned long long)(rejected ? 1 : 0));
            atomicAdd((unsigned long long*)&a.stats[2], count > 0 ? 1ull : 0ull);
            a.cursor[b] = n + count;
        }
        n_new = n + count;
        base = n;
        nrows = We + 1;
        __syncthreads();
    }
    // refresh the window for positions n_new+1 .. n_new+span
    if (n_new >= a.T) {
        if (t < W) {
            a.drafts[(size_t)b * W + t] = -1;
            a.qsrc[(size_t)b * W + t] = -1;
        }
        return;
    }
    const int span = min(W, a.T - n_new);
    const int reused = min(span, base + nrows - n_new);   // positions covered by this round's rows
    // reused predictions: the transform drew each row's candidate for the
    // position it predicts (u_draft of that position), or took its argmax
    for (int m = 1 + t; m <= reused; m += 256) {
        const int pos = n_new + m;
        const int prow = sl * R + (pos - base - 1);
        new_dr[m - 1] = a.greedy ? a.amax[prow] : a.samp[prow];
        new_q[m - 1] = prow;
    }
    __syncthreads();
    if (t == 0) {
        for (int m = reused + 1; m <= span; ++m) {
            const int pos = n_new + m;
            const int src = pos - a.H >= 1 ? pos - a.H : pos - 1;
            // both candidates are loaded from their own arrays and the value
            // selected, so neither access goes through a generic pointer
            const int from_x = a.xtok[(size_t)b * a.T + max(min(src, n_new) - 1, 0)];
            const int from_w = new_dr[max(src - n_new - 1, 0)];
            new_dr[m - 1] = src <= n_new ? from_x : from_w;
            new_q[m - 1] = -1;
        }
    }
    __syncthreads();
    if (t < W) {
        a.drafts[(size_t)b * W + t] = t < span ? new_dr[t] : -1;
        a.qsrc[(size_t)b * W + t] = t < span ? new_q[t] : -1;
    }
}

void verify_commit(const VerifyArgs& a, hipStream_t s) {
    if (a.nimg_cap <= 0) return;
    launch(k_verify, dim3(a.nimg_cap), dim3(256), 0, s, a);
}

// ---------------------------------------------------------------- state export
// q[i] = the proposal probability of draft i: its source row's p(z) for a
// reused prediction (qsrc >= 0) in probabilistic mode, 1 for a history draft
// (point mass) or in greedy mode, 0 where there is no draft
__global__ void k_gather_q(const float* __restrict__ P, const int32_t* __restrict__ qsrc,
                           const int32_t* __restrict__ drafts, int n, int V, int greedy,
                           float* __restrict__ q) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    const int z = drafts[i], qs = qsrc[i];
    float v = 0.f;
    if (z >= 0) v = (greedy || qs < 0) ? 1.0f : P[(size_t)qs * V + z];
    q[i] = v;
}

void gather_q(const float* P, const int32_t* qsrc, const int32_t* drafts, int n, int V,
              int greedy, float* q, hipStream_t s) {
    if (n <= 0) return;
    launch(k_gather_q, dim3((n + 255) / 256), dim3(256), 0, s, P, qsrc, drafts, n, V, greedy, q);
}

// ---------------------------------------------------------------- explicit-row transform
// Metadata of a transform over caller rows: row r is image r at sequence
// position pos[r] (clamped to [0, kRowPosMax]); the row's draw then uses
// u_draft(seed, r, pos[r]).
__global__ void k_transform_rows_setup(int rows, uint32_t seed_lo, uint32_t seed_hi,
                                       const int32_t* __restrict__ pos, int32_t* slot_img,
                                       int32_t* cursor, int32_t* meta) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < rows) {
        slot_img[i] = i;
        cursor[i] = min(max(pos[i], 0), kRowPosMax) - 1;
    }
    if (i < kMetaCount) {
        int v = 0;
        if (i == kMetaOutRows) v = rows;
        if (i == kMetaSeedLo) v = (int32_t)seed_lo;
        if (i == kMetaSeedHi) v = (int32_t)seed_hi;
        meta[i] = v;
    }
}

void transform_rows(int rows, int V, const float* logits, int cfg, float cfg_scale,
                    const float* temperature, int top_k, uint64_t seed, const int32_t* pos,
                    float* p, int32_t* amax, int32_t* draw, int32_t* scratch, hipStream_t s) {
    int32_t* slot_img = scratch;
    int32_t* cursor = scratch + rows;
    int32_t* meta = scratch + 2 * (size_t)rows;
    const int n = rows > kMetaCount ? rows : kMetaCount;
    launch(k_transform_rows_setup, dim3((n + 255) / 256), dim3(256), 0, s, rows, (uint32_t)seed,
           (uint32_t)(seed >> 32), pos, slot_img, cursor, meta);
    TransformArgs a{logits, p, amax, draw, slot_img, cursor, temperature, 1, cfg, V, top_k,
                    kRowPosMax, cfg_scale, meta + kMetaOutRows, rows, meta};
    transform(a, s);
}

// ---------------------------------------------------------------- explicit-row verification
__global__ __launch_bounds__(256) void k_verify_probs(int W, int V, const float* p, const float* q,
                                                      const int32_t* drafts, const float* u_acc,
                                                      const float* u_res, int32_t* counts,
                                                      int32_t* tokens) {
    __shared__ float cp[kMaxChunks + 1];
    __shared__ __attribute__((aligned(16))) float stage[kStageFloats];
    __shared__ int s_res, s_first;
    __shared__ int s_bad;
    const int b = blockIdx.x, t = threadIdx.x;
    if (t == 0) {
        s_first = W + 1;
        s_bad = 0;
    }
    __syncthreads();
    for (int j = t; j < W; j += 256) {
        const int z = drafts[(size_t)b * W + j];
        if (z < 0 || z >= V) s_bad = 1;
    }
    __syncthreads();
    if (s_bad) {
        for (int j = t; j < W; j += 256) tokens[(size_t)b * W + j] = -1;
        if (t == 0) counts[b] = 0;
        return;
    }
    for (int j = t; j < W; j += 256) {
        const size_t row = (size_t)b * W + j;
        const int z = drafts[row];
        const float P = p[row * V + z];
        const float Q = q[row * V + z];
        const bool acc = (P >= Q) || (u_acc[row] < P / Q);
        if (!acc) atomicMin(&s_first, j + 1);
    }
    __syncthreads();
    const int js = s_first;
    const bool rejected = js <= W;
    const int count = rejected ? js : W;
    int rep = 0;
    if (rejected) {
        const size_t row = (size_t)b * W + js - 1;
        rep = replacement_draw(p + row * V, q + row * V, drafts[row], V, u_res[b], stage, cp,
                               &s_res);
    }
    for (int j = t; j < W; j += 256) {
        const size_t row = (size_t)b * W + j;
        int tok = -1;
        if (j < count) tok = (j == count - 1 && rejected) ? rep : drafts[row];
        tokens[row] = tok;
    }
    if (t == 0) counts[b] = count;
}

void verify_probs(int B, int W, int V, const float* p, const float* q, const int32_t* drafts,
                  const float* u_acc, const float* u_res, int32_t* counts, int32_t* tokens,
                  hipStream_t s) {
    if (B <= 0) return;
    launch(k_verify_probs, dim3(B), dim3(256), 0, s, W, V, p, q, drafts, u_acc, u_res,
                       counts, tokens);
}

}  // namespace hbsjd
