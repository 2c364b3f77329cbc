// Causal attention of every sequence's window rows over its own paged KV cache
// (the batched verifier forward of Sec. 4.2: each image at its own position
// and KV location). Row i of a segment sits at position pos0 + i and attends to
// keys 0..pos0+i, which the QKV epilogue has already written (the window's own
// keys included).
//
// fp16 path (head_dim 64): one workgroup per (segment, query block, head); the
// four wavefronts split the 64-key tiles (= KV pages) round-robin by absolute
// tile index and run an online softmax on v_mfma_f32_16x16x32_f16 with the
// scores computed transposed, S^T = K Q^T: lane (g, c16) then owns query
// column c16 of each 16-query block, so the softmax needs only a two-step
// exchange across the four lane groups per block, and the probabilities are
// already laid out as the B operand of O^T = V^T P^T (V is stored transposed in
// the cache), so they never leave registers. The four partials are merged in a
// fixed order. A row's result therefore depends only on its position and the
// cache contents.
// fp32 path: one wavefront per (row, head), two-pass softmax.
#include <cstdlib>
#include <cstring>

#include "common.h"
#include "launch.h"

namespace hbsjd {

typedef __attribute__((ext_vector_type(8))) _Float16 f16x8_t;
typedef __attribute__((ext_vector_type(4))) float f32x4_t;

__device__ inline f16x8_t load_f16x8(const uint16_t* p) {
    return *reinterpret_cast<const f16x8_t*>(p);
}

template <int NMT>
__global__ __launch_bounds__(256) void k_attn_f16(const uint16_t* __restrict__ qb,
                                                   uint16_t* __restrict__ ob, int d, int H,
                                                   const uint16_t* __restrict__ kv, int maxp,
                                                   Segments seg, const int* __restrict__ nseg_dev,
                                                   int qblocks) {
    constexpr int QR = NMT * 16;   // query rows per block
    constexpr int LS = QR + 1;     // padded query stride of the parked partials
    const int sb = blockIdx.x, head = blockIdx.y;
    const int sg = sb / qblocks, qblk = sb - sg * qblocks;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int g = lane >> 4, c16 = lane & 15;
    // the segment's metadata, the count and the pages of this wavefront's first
    // two tiles are independent loads (the grid covers the segment capacity, and
    // the page list is indexed by segment), so they are in flight together
    const int nseg = *nseg_dev;
    const int nrows = seg.nrows[sg];
    const int row0s = seg.row0[sg];
    const int pos0 = seg.pos0[sg];
    const int page_a = seg.pages[(size_t)sg * maxp + min(w, maxp - 1)];
    const int page_b = seg.pages[(size_t)sg * maxp + min(w + 4, maxp - 1)];
    if (sg >= nseg) return;
    const int q0 = qblk * QR;
    if (q0 >= nrows) return;
    const int nq = min(QR, nrows - q0);
    const int row0 = row0s + q0;
    const int posf = pos0 + q0;
    const int ntiles = (posf + nq - 1) / 64 + 1;

    // wavefront w parks its partial O as [dim][query] in region w
    __shared__ float lds[4 * 64 * LS];
    __shared__ float mls[4][2][QR];

    // Q as the B operand: lane (g, c16) holds query c16 + 16 i, dims 32 kk + 8 g ..
    // (rows past the segment load its last row and are zeroed)
    f16x8_t qf[NMT][2];
#pragma unroll
    for (int i = 0; i < NMT; ++i) {
        const int r = i * 16 + c16;
        const int rr = min(r, nq - 1);
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
            const f16x8_t x = load_f16x8(qb + (size_t)(row0 + rr) * d + head * 64 + kk * 32 + 8 * g);
            qf[i][kk] = r < nq ? x : f16x8_t{};
        }
    }
    // O^T accumulators (dims dj*16 + 4 g + v of query c16 + 16 i), the column's
    // running maximum (equal in its four lanes) and this lane's share of the sum
    f32x4_t o[NMT][4];
    float m[NMT], l[NMT];
#pragma unroll
    for (int i = 0; i < NMT; ++i) {
        m[i] = -INFINITY;
        l[i] = 0.f;
#pragma unroll
        for (int dj = 0; dj < 4; ++dj) o[i][dj] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    }
    // K rows are fed in a permuted order: A-operand row c16 of 16-key group
    // j = 2 kk + h is key 32 kk + 8 (c16 >> 2) + 4 h + (c16 & 3). Score element
    // v of group j in lane (g, c16) is then key 32 kk + 8 g + 4 h + v, and the
    // eight scores of groups 2 kk, 2 kk + 1 are exactly the keys 32 kk + 8 g ..
    // + 7 that the B operand of the P V product needs in this lane.
    const int krow = 8 * (c16 >> 2) + (c16 & 3);
    const size_t page_elems = (size_t)2 * H * 64 * 64;
    for (int tile = w; tile < ntiles; tile += 4) {
        const int page = tile == w ? page_a
                         : tile == w + 4 ? page_b : seg.pages[(size_t)sg * maxp + tile];
        const uint16_t* Kb = kv + (size_t)page * page_elems + (size_t)head * 4096;
        const uint16_t* Vb = kv + (size_t)page * page_elems + (size_t)(H + head) * 4096;
        // both operands of the tile are fetched before any MFMA so their
        // latencies overlap
        f16x8_t kf[4][2], vf[4][2];
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int kd = 0; kd < 2; ++kd) {
                kf[j][kd] = load_f16x8(Kb + (32 * (j >> 1) + 4 * (j & 1) + krow) * 64 + kd * 32 + 8 * g);
                vf[j][kd] = load_f16x8(Vb + (j * 16 + c16) * 64 + kd * 32 + 8 * g);
            }
        f32x4_t s[NMT][4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
#pragma unroll
            for (int i = 0; i < NMT; ++i) s[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int kd = 0; kd < 2; ++kd)
#pragma unroll
                for (int i = 0; i < NMT; ++i)
                    s[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(kf[j][kd], qf[i][kd], s[i][j],
                                                                      0, 0, 0);
        }
        // online softmax of each query column over the tile's 64 keys
#pragma unroll
        for (int i = 0; i < NMT; ++i) {
            const int qr = i * 16 + c16;
            const int qpos = posf + qr;
            const bool qok = qr < nq;
            float mx = -INFINITY;
#pragma unroll
            for (int j = 0; j < 4; ++j)
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    const int key = tile * 64 + 32 * (j >> 1) + 8 * g + 4 * (j & 1) + v;
                    float x = s[i][j][v] * 0.125f;
                    if (!qok || key > qpos) x = -INFINITY;
                    s[i][j][v] = x;
                    mx = fmaxf(mx, x);
                }
            mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
            mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
            const float mnew = fmaxf(m[i], mx);
            const bool none = mnew == -INFINITY;
            const float alpha = none ? 1.f : __expf(m[i] - mnew);
            float ps = 0.f;
#pragma unroll
            for (int j = 0; j < 4; ++j)
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    const float pv = none ? 0.f : __expf(s[i][j][v] - mnew);
                    s[i][j][v] = pv;
                    ps += pv;
                }
            l[i] = l[i] * alpha + ps;
            m[i] = mnew;
#pragma unroll
            for (int dj = 0; dj < 4; ++dj) o[i][dj] *= alpha;
        }
        // O^T += V^T P^T, the B operand taken from this lane's own probabilities
#pragma unroll
        for (int kk = 0; kk < 2; ++kk)
#pragma unroll
            for (int i = 0; i < NMT; ++i) {
                f16x8_t pf;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    pf[e] = (_Float16)s[i][2 * kk][e];
                    pf[4 + e] = (_Float16)s[i][2 * kk + 1][e];
                }
#pragma unroll
                for (int dj = 0; dj < 4; ++dj)
                    o[i][dj] = __builtin_amdgcn_mfma_f32_16x16x32_f16(vf[dj][kk], pf, o[i][dj],
                                                                       0, 0, 0);
            }
    }
    // the column's sum over its four lanes
#pragma unroll
    for (int i = 0; i < NMT; ++i) {
        l[i] += __shfl_xor(l[i], 16, 64);
        l[i] += __shfl_xor(l[i], 32, 64);
    }
    // every wavefront parks its partial (o, m, l); a wavefront without tiles
    // parks m = -inf, l = 0
    float* Ow = lds + w * 64 * LS;
#pragma unroll
    for (int i = 0; i < NMT; ++i) {
#pragma unroll
        for (int dj = 0; dj < 4; ++dj)
#pragma unroll
            for (int v = 0; v < 4; ++v) Ow[(dj * 16 + 4 * g + v) * LS + i * 16 + c16] = o[i][dj][v];
        if (g == 0) {
            mls[w][0][i * 16 + c16] = m[i];
            mls[w][1][i * 16 + c16] = l[i];
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
        float lt = sc[0] * mls[0][1][r];
        for (int ww = 1; ww < 4; ++ww) {
            const float mw = mls[ww][0][r];
            sc[ww] = mw == -INFINITY ? 0.f : __expf(mw - ms);
            lt += sc[ww] * mls[ww][1][r];
        }
        float a = sc[0] * lds[lane * LS + r];
        for (int ww = 1; ww < 4; ++ww) a += sc[ww] * lds[ww * 64 * LS + lane * LS + r];
        ob[(size_t)(row0 + r) * d + head * 64 + lane] = f32_to_f16_rne(a / lt);
    }
}

// fp16, one wavefront per (segment, query block, head) when a launch has
// enough of them to fill the chip: the wavefront walks its keys' 64-key tiles
// in order with one online softmax and needs no LDS and no merge. With 16- and
// 32-query blocks the K and V fragments of tile t + 1 are in flight while tile
// t is multiplied; a 48-query block holds one tile at a time, which keeps it at
// two wavefronts per SIMD (XL rounds: 80 -> 63 us, the bits unchanged). The
// score and probability layouts are those of k_attn_f16 (S^T = K Q^T,
// O^T = V^T P^T). A row's result depends only on its position and the cache.
template <int NMT>
__global__ __launch_bounds__(64) void k_attn_f16_seq(const uint16_t* __restrict__ qb,
                                                     uint16_t* __restrict__ ob, int d, int H,
                                                     const uint16_t* __restrict__ kv, int maxp,
                                                     Segments seg, const int* __restrict__ nseg_dev,
                                                     int qblocks) {
    constexpr int QR = NMT * 16;
    const int sb = blockIdx.x, head = blockIdx.y;
    const int sg = sb / qblocks, qblk = sb - sg * qblocks;
    const int lane = threadIdx.x;
    const int g = lane >> 4, c16 = lane & 15;
    const int nseg = *nseg_dev;
    const int nrows = seg.nrows[sg];
    const int row0s = seg.row0[sg];
    const int pos0 = seg.pos0[sg];
    // the segment's page list, one entry per lane (maxp <= 64)
    const int pagev = seg.pages[(size_t)sg * maxp + min(lane, maxp - 1)];
    if (sg >= nseg) return;
    const int q0 = qblk * QR;
    if (q0 >= nrows) return;
    const int nq = min(QR, nrows - q0);
    const int row0 = row0s + q0;
    const int posf = pos0 + q0;
    const int ntiles = (posf + nq - 1) / 64 + 1;

    f16x8_t qf[NMT][2];
#pragma unroll
    for (int i = 0; i < NMT; ++i) {
        const int r = i * 16 + c16;
        const int rr = min(r, nq - 1);
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
            const f16x8_t x = load_f16x8(qb + (size_t)(row0 + rr) * d + head * 64 + kk * 32 + 8 * g);
            qf[i][kk] = r < nq ? x : f16x8_t{};
        }
    }
    f32x4_t o[NMT][4];
    float m[NMT], l[NMT];
#pragma unroll
    for (int i = 0; i < NMT; ++i) {
        m[i] = -INFINITY;
        l[i] = 0.f;
#pragma unroll
        for (int dj = 0; dj < 4; ++dj) o[i][dj] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    }
    const int krow = 8 * (c16 >> 2) + (c16 & 3);
    const size_t page_elems = (size_t)2 * H * 64 * 64;
    // K and V fragments of one tile (the page of tile t is lane t's entry)
    auto fetch = [&](int tile, f16x8_t (&kf)[4][2], f16x8_t (&vf)[4][2]) {
        const int page = __builtin_amdgcn_readlane(pagev, tile);
        const uint16_t* Kb = kv + (size_t)page * page_elems + (size_t)head * 4096;
        const uint16_t* Vb = kv + (size_t)page * page_elems + (size_t)(H + head) * 4096;
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int kd = 0; kd < 2; ++kd) {
                kf[j][kd] = load_f16x8(Kb + (32 * (j >> 1) + 4 * (j & 1) + krow) * 64 + kd * 32 + 8 * g);
                vf[j][kd] = load_f16x8(Vb + (j * 16 + c16) * 64 + kd * 32 + 8 * g);
            }
    };
    // scores in log2 units: y = (q . k) / 8 * log2(e), p = 2^(y - max); rows
    // past the segment (q = 0) are computed and never stored
    constexpr float kScale = 0.125f * 1.44269504088896340736f;
    auto tile_step = [&](int tile, const f16x8_t (&kf)[4][2], const f16x8_t (&vf)[4][2]) {
        f32x4_t s[NMT][4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
#pragma unroll
            for (int i = 0; i < NMT; ++i) s[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int kd = 0; kd < 2; ++kd)
#pragma unroll
                for (int i = 0; i < NMT; ++i)
                    s[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(kf[j][kd], qf[i][kd], s[i][j],
                                                                      0, 0, 0);
        }
#pragma unroll
        for (int i = 0; i < NMT; ++i) {
            // element v of group j is key tile * 64 + 32 (j >> 1) + 8 g + 4 (j & 1) + v,
            // visible while v <= lim - 32 (j >> 1) - 4 (j & 1)
            const int lim = posf + i * 16 + c16 - tile * 64 - 8 * g;
            float mx = -INFINITY;
#pragma unroll
            for (int j = 0; j < 4; ++j)
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    float x = s[i][j][v] * kScale;
                    if (v > lim - 32 * (j >> 1) - 4 * (j & 1)) x = -INFINITY;
                    s[i][j][v] = x;
                    mx = fmaxf(mx, x);
                }
            mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
            mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
            // tile 0 holds key 0, which every row sees: the maximum is finite
            // from the first tile on
            const float mnew = fmaxf(m[i], mx);
            const float alpha = exp2f(m[i] - mnew);
            float ps = 0.f;
#pragma unroll
            for (int j = 0; j < 4; ++j)
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    const float pv = exp2f(s[i][j][v] - mnew);
                    s[i][j][v] = pv;
                    ps += pv;
                }
            l[i] = l[i] * alpha + ps;
            m[i] = mnew;
#pragma unroll
            for (int dj = 0; dj < 4; ++dj) o[i][dj] *= alpha;
        }
#pragma unroll
        for (int kk = 0; kk < 2; ++kk)
#pragma unroll
            for (int i = 0; i < NMT; ++i) {
                f16x8_t pf;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    pf[e] = (_Float16)s[i][2 * kk][e];
                    pf[4 + e] = (_Float16)s[i][2 * kk + 1][e];
                }
#pragma unroll
                for (int dj = 0; dj < 4; ++dj)
                    o[i][dj] = __builtin_amdgcn_mfma_f32_16x16x32_f16(vf[dj][kk], pf, o[i][dj],
                                                                       0, 0, 0);
            }
    };
    if constexpr (NMT >= 3) {
        for (int tile = 0; tile < ntiles; ++tile) {
            f16x8_t kc[4][2], vc[4][2];
            fetch(tile, kc, vc);
            tile_step(tile, kc, vc);
        }
    } else {
        // two register buffers; every fetch is issued (the last tile
        // re-fetched past the end), so the loads in flight are the same on
        // every path
        f16x8_t ka[4][2], va[4][2], kb[4][2], vb[4][2];
        fetch(0, ka, va);
        for (int tile = 0; tile < ntiles; tile += 2) {
            fetch(min(tile + 1, ntiles - 1), kb, vb);
            tile_step(tile, ka, va);
            if (tile + 1 >= ntiles) break;
            fetch(min(tile + 2, ntiles - 1), ka, va);
            tile_step(tile + 1, kb, vb);
        }
    }
#pragma unroll
    for (int i = 0; i < NMT; ++i) {
        l[i] += __shfl_xor(l[i], 16, 64);
        l[i] += __shfl_xor(l[i], 32, 64);
    }
    // lane (g, c16) holds dims dj * 16 + 4 g .. + 3 of query c16 + 16 i: four
    // halves per store
#pragma unroll
    for (int i = 0; i < NMT; ++i) {
        const int qr = i * 16 + c16;
        if (qr >= nq) continue;
        uint16_t* dst = ob + (size_t)(row0 + qr) * d + head * 64 + 4 * g;
#pragma unroll
        for (int dj = 0; dj < 4; ++dj) {
            uint32_t w0 = f32_to_f16_rne(o[i][dj][0] / l[i]) | ((uint32_t)f32_to_f16_rne(o[i][dj][1] / l[i]) << 16);
            uint32_t w1 = f32_to_f16_rne(o[i][dj][2] / l[i]) | ((uint32_t)f32_to_f16_rne(o[i][dj][3] / l[i]) << 16);
            *reinterpret_cast<uint2*>(dst + dj * 16) = make_uint2(w0, w1);
        }
    }
}

// fp16, one workgroup of four wavefronts per (segment, head) for segments of
// at most 64 rows: wavefront w takes query rows 16 w .. 16 w + 15, and all
// four stream the segment's K and V^T tiles through two LDS buffers with
// direct loads (global_load_lds_dwordx4), tile t + 1's loads issued while
// tile t is multiplied. Prefetch then costs LDS instead of registers (87
// VGPRs, five workgroups per CU), and each tile leaves memory once for every
// query block. (Walking two or four heads per workgroup as one stream, so the
// next head's first tile is in flight too, measured slower: fewer
// workgroups.) Every wavefront walks the tiles up to the segment's last row,
// as a 48-row block of k_attn_f16_seq does, with the same per-row arithmetic,
// so rows come out bit-identical to it. LDS rows hold eight 16-byte chunks;
// chunk c of row r sits at c ^ f(r), with f chosen so that the eight lanes of
// a fragment read land on eight different chunk positions: K rows are read in
// the permuted order of the score layout (rows 8a + b, b < 4, together),
// f(r) = (r & 3) | ((r >> 1) & 4); V^T rows are read consecutively,
// f(r) = r & 7.
__device__ __forceinline__ int qs_swz_k(int r) { return (r & 3) | ((r >> 1) & 4); }
__device__ __forceinline__ int qs_swz_v(int r) { return r & 7; }

__global__ __launch_bounds__(256) void k_attn_f16_qs(const uint16_t* __restrict__ qb,
                                                     uint16_t* __restrict__ ob, int d, int H,
                                                     const uint16_t* __restrict__ kv, int maxp,
                                                     Segments seg, const int* __restrict__ nseg_dev) {
    // [buffer][K, V^T][64 rows x 64], 32 KB
    __shared__ __attribute__((aligned(1024))) uint16_t kvs[2][2][64 * 64];
    const int sg = blockIdx.x, head = blockIdx.y;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int g = lane >> 4, c16 = lane & 15;
    const int nseg = *nseg_dev;
    const int nrows = seg.nrows[sg];
    const int row0s = seg.row0[sg];
    const int pos0 = seg.pos0[sg];
    const int pagev = seg.pages[(size_t)sg * maxp + min(lane, maxp - 1)];
    if (sg >= nseg || nrows <= 0) return;   // the whole workgroup
    const int ntiles = (pos0 + nrows - 1) / 64 + 1;
    const int q0 = 16 * w;
    const int nq = min(16, nrows - q0);   // <= 0: this wavefront only loads
    const int posf = pos0 + q0;
    const size_t page_elems = (size_t)2 * H * 64 * 64;

    // wavefront w loads 1 KB blocks w, w + 4, w + 8, w + 12 of a tile (blocks
    // 0-7 K rows, 8-15 V^T rows, 8 rows each): lane l's chunk lands at 16 l
    // bytes into the block, LDS row 8 (b & 7) + (l >> 3), position l & 7
    auto issue = [&](int tile, int buf) {
        const int page = __builtin_amdgcn_readlane(pagev, tile);
        const uint16_t* base = kv + (size_t)page * page_elems + (size_t)head * 4096;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int b = w + 4 * k;
            const int part = b >> 3, r = 8 * (b & 7) + (lane >> 3);
            const int c = (lane & 7) ^ (part == 0 ? qs_swz_k(r) : qs_swz_v(r));
            const uint16_t* src = base + (size_t)part * H * 4096 + r * 64 + c * 8;
            load_to_lds16(src, &kvs[buf][part][(b & 7) * 512]);
        }
    };
    f16x8_t qf[2];
    f32x4_t o[4];
    float m = -INFINITY, l = 0.f;
    if (nq > 0) {
        const int rr = min(c16, nq - 1);
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
            const f16x8_t x = load_f16x8(qb + (size_t)(row0s + q0 + rr) * d + head * 64 + kk * 32 + 8 * g);
            qf[kk] = c16 < nq ? x : f16x8_t{};
        }
    }
#pragma unroll
    for (int dj = 0; dj < 4; ++dj) o[dj] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    const int krow = 8 * (c16 >> 2) + (c16 & 3);
    constexpr float kScale = 0.125f * 1.44269504088896340736f;

    issue(0, 0);
    for (int tile = 0; tile < ntiles; ++tile) {
        wait_loads<0>();
        lds_barrier();   // tile's loads landed everywhere; the other buffer is free
        if (tile + 1 < ntiles) issue(tile + 1, (tile + 1) & 1);
        if (nq <= 0) continue;
        const uint16_t* Ks = kvs[tile & 1][0];
        const uint16_t* Vs = kvs[tile & 1][1];
        f32x4_t s[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            s[j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
            const int r = 32 * (j >> 1) + 4 * (j & 1) + krow;
#pragma unroll
            for (int kd = 0; kd < 2; ++kd) {
                const f16x8_t kf = load_f16x8(Ks + r * 64 + (((kd * 4 + g) ^ qs_swz_k(r)) << 3));
                s[j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(kf, qf[kd], s[j], 0, 0, 0);
            }
        }
        // as in k_attn_f16_seq: element v of group j is key tile * 64 +
        // 32 (j >> 1) + 8 g + 4 (j & 1) + v, visible while
        // v <= lim - 32 (j >> 1) - 4 (j & 1)
        const int lim = posf + c16 - tile * 64 - 8 * g;
        float mx = -INFINITY;
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                float x = s[j][v] * kScale;
                if (v > lim - 32 * (j >> 1) - 4 * (j & 1)) x = -INFINITY;
                s[j][v] = x;
                mx = fmaxf(mx, x);
            }
        mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
        mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
        const float mnew = fmaxf(m, mx);
        const float alpha = exp2f(m - mnew);
        float ps = 0.f;
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const float pv = exp2f(s[j][v] - mnew);
                s[j][v] = pv;
                ps += pv;
            }
        l = l * alpha + ps;
        m = mnew;
#pragma unroll
        for (int dj = 0; dj < 4; ++dj) o[dj] *= alpha;
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
            f16x8_t pf;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                pf[e] = (_Float16)s[2 * kk][e];
                pf[4 + e] = (_Float16)s[2 * kk + 1][e];
            }
#pragma unroll
            for (int dj = 0; dj < 4; ++dj) {
                const int r = dj * 16 + c16;
                const f16x8_t vf = load_f16x8(Vs + r * 64 + (((kk * 4 + g) ^ qs_swz_v(r)) << 3));
                o[dj] = __builtin_amdgcn_mfma_f32_16x16x32_f16(vf, pf, o[dj], 0, 0, 0);
            }
        }
    }
    if (nq <= 0) return;
    l += __shfl_xor(l, 16, 64);
    l += __shfl_xor(l, 32, 64);
    if (c16 >= nq) return;
    uint16_t* dst = ob + (size_t)(row0s + q0 + c16) * d + head * 64 + 4 * g;
#pragma unroll
    for (int dj = 0; dj < 4; ++dj) {
        uint32_t w0 = f32_to_f16_rne(o[dj][0] / l) | ((uint32_t)f32_to_f16_rne(o[dj][1] / l) << 16);
        uint32_t w1 = f32_to_f16_rne(o[dj][2] / l) | ((uint32_t)f32_to_f16_rne(o[dj][3] / l) << 16);
        *reinterpret_cast<uint2*>(dst + dj * 16) = make_uint2(w0, w1);
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

// HBSJD_ATTN_KERNEL: 2 "qs" (else "seq"), 1 "seq", -1 "split", 0 chosen per launch
static int g_force_attn = 0;

void attention_setup() {
    const char* f = std::getenv("HBSJD_ATTN_KERNEL");
    g_force_attn = !f ? 0 : std::strcmp(f, "qs") == 0 ? 2 : std::strcmp(f, "seq") == 0 ? 1
                 : std::strcmp(f, "split") == 0 ? -1 : 0;
}

void attention(bool f16, const void* q, void* o, int d, int heads, int head_dim,
               const void* kv_layer, const int32_t* ptab, int max_pages, const Segments& seg,
               const int* nseg_dev, int nseg_cap, int max_rows_per_seg, const RowMeta& rows,
               const int* nrows_dev, int nrows_cap, hipStream_t s) {
    if (f16) {
        if (nseg_cap <= 0) return;
        // Segments of at most 64 rows (every round) whose launch has at least
        // 512 (segment, head) pairs take k_attn_f16_qs; longer segments (the
        // prefill) take one wavefront per (segment, query block, head) once
        // the launch has at least 2048 of them (8 per CU). Both need the page
        // list to fit a wavefront. Below that, four wavefronts split each
        // block's keys. The choice depends only on the launch's capacities, so
        // Full and Compact rounds take the same kernel. (HBSJD_ATTN_KERNEL
        // forces one kernel for every launch it fits, for tests; "qs" takes
        // the sequential kernel where the query-split one does not fit.)
        const int rows_blk = max_rows_per_seg <= 16 ? 16 : max_rows_per_seg <= 32 ? 32
                           : max_rows_per_seg <= 48 ? 48 : 32;
        const int qbl = (max_rows_per_seg + rows_blk - 1) / rows_blk;
        const bool seq_ok = max_pages <= 64;
        const bool qs_ok = seq_ok && max_rows_per_seg <= 64;
        const bool take_qs = g_force_attn == 2 ? qs_ok
                           : g_force_attn != 0 ? false
                           : qs_ok && (long)nseg_cap * heads >= 512;
        if (take_qs) {
            launch(k_attn_f16_qs, dim3(nseg_cap, heads), dim3(256), 0, s, (const uint16_t*)q,
                   (uint16_t*)o, d, heads, (const uint16_t*)kv_layer, max_pages, seg, nseg_dev);
            return;
        }
        const bool take_seq = g_force_attn >= 1 ? seq_ok
                            : g_force_attn < 0 ? false
                            : (long)nseg_cap * qbl * heads >= 2048 && seq_ok;
        if (take_seq) {
            const dim3 grid(nseg_cap * qbl, heads);
            if (rows_blk == 16)
                launch(k_attn_f16_seq<1>, grid, dim3(64), 0, s, (const uint16_t*)q, (uint16_t*)o, d,
                       heads, (const uint16_t*)kv_layer, max_pages, seg, nseg_dev, qbl);
            else if (rows_blk == 48)
                launch(k_attn_f16_seq<3>, grid, dim3(64), 0, s, (const uint16_t*)q, (uint16_t*)o, d,
                       heads, (const uint16_t*)kv_layer, max_pages, seg, nseg_dev, qbl);
            else
                launch(k_attn_f16_seq<2>, grid, dim3(64), 0, s, (const uint16_t*)q, (uint16_t*)o, d,
                       heads, (const uint16_t*)kv_layer, max_pages, seg, nseg_dev, qbl);
            return;
        }
        if (max_rows_per_seg <= 16) {
            launch(k_attn_f16<1>, dim3(nseg_cap, heads), dim3(256), 0, s, (const uint16_t*)q,
                   (uint16_t*)o, d, heads, (const uint16_t*)kv_layer, max_pages, seg, nseg_dev, 1);
        } else if (max_rows_per_seg > 32 && max_rows_per_seg <= 48) {
            // a round window of 33..48 rows in one block, so the sequence's
            // keys and values are read once per head (two 32-row blocks would
            // each read them)
            launch(k_attn_f16<3>, dim3(nseg_cap, heads), dim3(256), 0, s, (const uint16_t*)q,
                   (uint16_t*)o, d, heads, (const uint16_t*)kv_layer, max_pages, seg, nseg_dev, 1);
        } else {
            // 32 query rows per block; long (prefill) segments split into several
            const int qblocks = (max_rows_per_seg + 31) / 32;
            launch(k_attn_f16<2>, dim3(nseg_cap * qblocks, heads), dim3(256), 0, s,
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
