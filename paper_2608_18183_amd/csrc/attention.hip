// Causal attention of every sequence's window rows over its own paged KV cache
// (the batched verifier forward of Sec. 4.2: each image at its own position
// and KV location). Row i of a segment sits at position pos0 + i and attends to
// keys 0..pos0+i, which the QKV epilogue has already written (the window's own
// keys included).
//
// bf16 path (head_dim 64): one workgroup per (segment, query block, head); the
// four wavefronts split the 64-key tiles (= KV pages) round-robin by absolute
// tile index, run an online softmax with S = Q K^T and O += P V on
// v_mfma_f32_16x16x32_bf16, and merge their partials in a fixed order. A row's
// result therefore depends only on its position and the cache contents.
// fp32 path: one wavefront per (row, head), two-pass softmax.
#include "common.h"
#include "launch.h"

namespace hbsjd {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(4))) float f32x4_t;

__device__ inline bf16x8_t load_bf16x8(const uint16_t* p) {
    return *reinterpret_cast<const bf16x8_t*>(p);
}

template <int NMT>
__global__ __launch_bounds__(256) void k_attn_bf16(const uint16_t* __restrict__ qb,
                                                   uint16_t* __restrict__ ob, int d, int H,
                                                   const uint16_t* __restrict__ kv, int maxp,
                                                   Segments seg, const int* __restrict__ nseg_dev,
                                                   int qblocks) {
    constexpr int QR = NMT * 16;   // query rows per block
    const int sb = blockIdx.x, head = blockIdx.y;
    const int sg = sb / qblocks, qblk = sb - sg * qblocks;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int g = lane >> 4, c16 = lane & 15;
    // the segment's metadata, the count and this wavefront's first page are
    // independent loads (the grid covers the segment capacity, and the page
    // list is indexed by segment), so they are in flight together
    const int nseg = *nseg_dev;
    const int nrows = seg.nrows[sg];
    const int row0s = seg.row0[sg];
    const int pos0 = seg.pos0[sg];
    const int page_w = seg.pages[(size_t)sg * maxp + min(w, maxp - 1)];
    if (sg >= nseg) return;
    const int q0 = qblk * QR;
    if (q0 >= nrows) return;
    const int nq = min(QR, nrows - q0);
    const int row0 = row0s + q0;
    const int posf = pos0 + q0;
    const int ntiles = (posf + nq - 1) / 64 + 1;

    // LDS: wavefront w owns region w (QR x 64 floats): P (bf16) during the tile
    // loop, then its partial output for the merge
    __shared__ __attribute__((aligned(16))) float lds[4 * QR * 64];
    __shared__ float mls[4][2][QR];
    float* Ow = lds + w * QR * 64;
    uint16_t* Pw = reinterpret_cast<uint16_t*>(Ow);

    bf16x8_t qf[NMT][2];
#pragma unroll
    for (int i = 0; i < NMT; ++i) {
        const int r = i * 16 + c16;
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
            if (r < nq)
                qf[i][kk] = load_bf16x8(qb + (size_t)(row0 + r) * d + head * 64 + kk * 32 + 8 * g);
            else
                qf[i][kk] = bf16x8_t{};
        }
    }
    f32x4_t o[NMT][4];
    float mrow[NMT][4], lrow[NMT][4];
#pragma unroll
    for (int i = 0; i < NMT; ++i)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            mrow[i][v] = -INFINITY;
            lrow[i][v] = 0.f;
            o[i][v] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        }

    const size_t page_elems = (size_t)2 * H * 64 * 64;
    for (int tile = w; tile < ntiles; tile += 4) {
        const int page = tile == w ? page_w : seg.pages[(size_t)sg * maxp + tile];
        const uint16_t* Kb = kv + (size_t)page * page_elems + (size_t)head * 4096;
        const uint16_t* Vb = kv + (size_t)page * page_elems + (size_t)(H + head) * 4096;
        // both operands of the tile are fetched before any MFMA so their
        // latencies overlap
        bf16x8_t kf[4][2], vf[4][2];
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int kk = 0; kk < 2; ++kk) {
                kf[j][kk] = load_bf16x8(Kb + (j * 16 + c16) * 64 + kk * 32 + 8 * g);
                vf[j][kk] = load_bf16x8(Vb + (j * 16 + c16) * 64 + kk * 32 + 8 * g);
            }
        f32x4_t s[NMT][4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
#pragma unroll
            for (int i = 0; i < NMT; ++i) s[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int kk = 0; kk < 2; ++kk)
#pragma unroll
                for (int i = 0; i < NMT; ++i)
                    s[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qf[i][kk], kf[j][kk], s[i][j],
                                                                      0, 0, 0);
        }
        // online softmax; lane holds rows 4g+v of key columns c16 + 16 j
#pragma unroll
        for (int i = 0; i < NMT; ++i) {
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int r = i * 16 + 4 * g + v;
                const int qpos = posf + r;
                float mx = -INFINITY;
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int key = tile * 64 + j * 16 + c16;
                    float x = s[i][j][v] * 0.125f;
                    if (r >= nq || key > qpos) x = -INFINITY;
                    s[i][j][v] = x;
                    mx = fmaxf(mx, x);
                }
                mx = fmaxf(mx, __shfl_xor(mx, 1, 64));
                mx = fmaxf(mx, __shfl_xor(mx, 2, 64));
                mx = fmaxf(mx, __shfl_xor(mx, 4, 64));
                mx = fmaxf(mx, __shfl_xor(mx, 8, 64));
                const float mnew = fmaxf(mrow[i][v], mx);
                const bool none = mnew == -INFINITY;
                const float alpha = none ? 1.f : __expf(mrow[i][v] - mnew);
                float ps = 0.f;
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const float pv = none ? 0.f : __expf(s[i][j][v] - mnew);
                    s[i][j][v] = pv;
                    ps += pv;
                }
                ps += __shfl_xor(ps, 1, 64);
                ps += __shfl_xor(ps, 2, 64);
                ps += __shfl_xor(ps, 4, 64);
                ps += __shfl_xor(ps, 8, 64);
                lrow[i][v] = lrow[i][v] * alpha + ps;
                mrow[i][v] = mnew;
#pragma unroll
                for (int dj = 0; dj < 4; ++dj) o[i][dj][v] *= alpha;
            }
        }
        // P (bf16) to this wave's LDS region as [row][key], read back as A operand
#pragma unroll
        for (int i = 0; i < NMT; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j)
#pragma unroll
                for (int v = 0; v < 4; ++v)
                    Pw[(i * 16 + 4 * g + v) * 64 + j * 16 + c16] = f32_to_bf16(s[i][j][v]);
        // P was written by other lanes of this wavefront: order the LDS writes
        // before the reads below at wavefront scope
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
            bf16x8_t pf[NMT];
#pragma unroll
            for (int i = 0; i < NMT; ++i)
                pf[i] = *reinterpret_cast<const bf16x8_t*>(Pw + (i * 16 + c16) * 64 + kk * 32 + 8 * g);
#pragma unroll
            for (int dj = 0; dj < 4; ++dj) {
#pragma unroll
                for (int i = 0; i < NMT; ++i)
                    o[i][dj] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pf[i], vf[dj][kk], o[i][dj],
                                                                       0, 0, 0);
            }
        }
        // the next tile (or the partial below) overwrites P: keep those writes
        // after these reads
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }
    // every wavefront parks its partial (o, m, l); a wavefront without tiles
    // parks m = -inf, l = 0
#pragma unroll
    for (int i = 0; i < NMT; ++i)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int r = i * 16 + 4 * g + v;
#pragma unroll
            for (int dj = 0; dj < 4; ++dj) Ow[r * 64 + dj * 16 + c16] = o[i][dj][v];
            if (c16 == 0) {
                mls[w][0][r] = mrow[i][v];
                mls[w][1][r] = lrow[i][v];
            }
        }
    __syncthreads();
    // merge the four partials in wave order 0, 1, 2, 3 (tile 0 is wave 0's, so
    // its maximum is finite); wavefront w merges rows w, w + 4, ..., lane = dim
    for (int r = w; r < nq; r += 4) {
        const float m0 = mls[0][0][r];
        float ms = m0;
        for (int ww = 1; ww < 4; ++ww) ms = fmaxf(ms, mls[ww][0][r]);
        float sc[4];
        sc[0] = __expf(m0 - ms);
        float l = sc[0] * mls[0][1][r];
        for (int ww = 1; ww < 4; ++ww) {
            const float mw = mls[ww][0][r];
            sc[ww] = mw == -INFINITY ? 0.f : __expf(mw - ms);
            l += sc[ww] * mls[ww][1][r];
        }
        const float inv = 1.0f / l;
        float a = sc[0] * lds[r * 64 + lane];
        for (int ww = 1; ww < 4; ++ww) a += sc[ww] * lds[ww * QR * 64 + r * 64 + lane];
        ob[(size_t)(row0 + r) * d + head * 64 + lane] = f32_to_bf16(a * inv);
    }
}

// fp32: one wavefront per (row, head); scores over keys 0..pos in LDS.
__global__ __launch_bounds__(64) void k_attn_f32(const float* __restrict__ q,
                                                 float* __restrict__ o, int d, int H, int dh,
                                                 const float* __restrict__ kv,
                                                 const int32_t* __restrict__ ptab, int maxp,
                                                 RowMeta rows, const int* __restrict__ nrows_dev) {
    __shared__ float sc[1024];
    __shared__ float qs[64];
    const int r = blockIdx.x, head = blockIdx.y, lane = threadIdx.x;
    if (r >= *nrows_dev) return;
    const int pos = rows.pos[r], sq = rows.seq[r];
    if (lane < dh) qs[lane] = q[(size_t)r * d + head * dh + lane];
    __syncthreads();
    const float scale = 1.0f / sqrtf((float)dh);
    const size_t page_elems = (size_t)2 * H * 64 * dh;
    float mx = -INFINITY;
    for (int j = lane; j <= pos; j += 64) {
        const int page = ptab[(size_t)sq * maxp + (j >> 6)];
        const float* kr = kv + (size_t)page * page_elems + (size_t)head * 64 * dh + (size_t)(j & 63) * dh;
        float acc = 0.f;
        for (int e = 0; e < dh; ++e) acc = fmaf(qs[e], kr[e], acc);
        acc *= scale;
        sc[j] = acc;
        mx = fmaxf(mx, acc);
    }
    mx = wave_max(mx);
    float z = 0.f;
    for (int j = lane; j <= pos; j += 64) {
        const float e = expf(sc[j] - mx);
        sc[j] = e;
        z += e;
    }
    z = wave_sum(z);
    __syncthreads();
    if (lane < dh) {
        float acc = 0.f;
        for (int j = 0; j <= pos; ++j) {
            const int page = ptab[(size_t)sq * maxp + (j >> 6)];
            const float* vt = kv + (size_t)page * page_elems + (size_t)(H + head) * 64 * dh;
            acc = fmaf(sc[j] / z, vt[(size_t)lane * 64 + (j & 63)], acc);
        }
        o[(size_t)r * d + head * dh + lane] = acc;
    }
}

void attention(bool bf16, const void* q, void* o, int d, int heads, int head_dim,
               const void* kv_layer, const int32_t* ptab, int max_pages, const Segments& seg,
               const int* nseg_dev, int nseg_cap, int max_rows_per_seg, const RowMeta& rows,
               const int* nrows_dev, int nrows_cap, hipStream_t s) {
    if (bf16) {
        if (nseg_cap <= 0) return;
        if (max_rows_per_seg <= 16) {
            launch(k_attn_bf16<1>, dim3(nseg_cap, heads), dim3(256), 0, s, (const uint16_t*)q,
                   (uint16_t*)o, d, heads, (const uint16_t*)kv_layer, max_pages, seg, nseg_dev, 1);
        } else {
            // 32 query rows per block; long (prefill) segments split into several
            const int qblocks = (max_rows_per_seg + 31) / 32;
            launch(k_attn_bf16<2>, dim3(nseg_cap * qblocks, heads), dim3(256), 0, s,
                   (const uint16_t*)q, (uint16_t*)o, d, heads, (const uint16_t*)kv_layer,
                   max_pages, seg, nseg_dev, qblocks);
        }
    } else {
        if (nrows_cap <= 0) return;
        launch(k_attn_f32, dim3(nrows_cap, heads), dim3(64), 0, s, (const float*)q,
                           (float*)o, d, heads, head_dim, (const float*)kv_layer, ptab, max_pages,
                           rows, nrows_dev);
    }
}

}  // namespace hbsjd
