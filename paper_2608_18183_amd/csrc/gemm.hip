// Dense contractions of the verifier forward: QKV, O, W1|W3 and W2 projections
// and the lm_head, each C = A . W^T with the neighbouring elementwise work
// fused into the epilogue (2D RoPE and the paged KV append after QKV, the
// residual add after O and W2, SwiGLU after W1|W3, bias after the lm_head).
//
// fp16 path (the bf16 model's weights held as scaled fp16, fp16 activations):
// 256-thread workgroups, 2x2 wavefronts, LDS-staged 64-deep K tiles with an
// XOR swizzle (loaded straight into LDS for the 64x64 tile, through registers
// for the 128x128 one), v_mfma_f32_16x16x32_f16 with fp32 accumulation, the
// sums multiplied by the weights' inverse scale before the epilogue. An output
// element sums its K range in the same order wherever its row sits in the launch, and for the unsplit projections (QKV, W1|W3,
// lm_head) whatever the launch's size or tile. O and W2 cut K into as many
// parts as split_for gives for the launch's row capacity, so there the order
// of the partial sums, and a row's last bits, follow that capacity.
// fp32 path: a plain LDS-tiled FMA kernel for the exact-parity mode.
#include "common.h"
#include "launch.h"

#include <algorithm>
#include <cstdlib>
#include <cstring>
#include <map>
#include <mutex>

// Elementwise epilogue arithmetic rounds every operation on its own (no fused
// multiply-add contraction), so the wide-tile and the smaller-tile kernels,
// whose epilogue code differs, give the same bits for the same row
#pragma clang fp contract(off)

namespace hbsjd {

typedef __attribute__((ext_vector_type(8))) _Float16 f16x8_t;
typedef __attribute__((ext_vector_type(4))) float f32x4_t;
// 16-byte staging chunk as a first-class vector (a copy of HIP's uint4 struct
// becomes a memcpy that keeps the stage arrays out of registers)
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4_t;

// the value lane l ^ 1 holds (DPP quad permutation [1, 0, 3, 2])
__device__ __forceinline__ float swap_lane_pair(float v) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0xB1, 0xF, 0xF, false));
}

// ---------------------------------------------------------------- epilogues
// operator()(row, col, value, value of column col ^ 1 in the same row)

// The fp16 kernel calls begin_tile(n0) once, row_info(m) once per output row
// and operator()(info, m, n, value, partner) per element; the fp32 kernel only
// uses the last two.

// 2D RoPE of one pair (x0, x1) = (element 2i, element 2i+1) of a head:
// (x0 cos - x1 sin, x0 sin + x1 cos), each product rounded on its own (this
// file compiles without contraction), so every kernel that applies it gets
// the same bits
__device__ __forceinline__ float rope_even(float x0, float x1, float cs, float sn) {
    return x0 * cs - x1 * sn;
}
__device__ __forceinline__ float rope_odd(float x0, float x1, float cs, float sn) {
    return x0 * sn + x1 * cs;
}

template <typename T>
struct EpiQkv {
    T* q;
    T* kv;
    const int32_t* pos;
    const int32_t* kvslot;
    const float* rc;
    const float* rs;
    int d, heads, dh, T_;
    int part = 0;   // 0 q, 1 k, 2 v: fixed per tile since d is a multiple of the tile width
    // the fp16 path has head_dim 64; the fp32 path takes it at run time
    static constexpr int kDh = sizeof(T) == 2 ? 64 : 0;
    // the RoPE factors are fetched after the main loop: holding them through it
    // costs more (register pressure) than the one exposed load
    static constexpr bool kLateAux = true;
    __device__ int head_dim() const { return kDh ? kDh : dh; }
    // element offsets are 32-bit (the host keeps every activation buffer and a
    // layer's KV pool below 2^31 elements). A row carries its position and the
    // offset of its entry for this tile's part (q row; K slot of head 0; V^T
    // column of head 0), so an element only adds its column part.
    struct Row { int p, off; };
    struct Aux { float cs, sn; };
    __device__ void begin_tile(int n0) { part = n0 / d; }
    __device__ Row row_info(int m) const {
        const int p = pos[m], slot = kvslot[m];
        const int dhv = head_dim();
        const int page = slot >> 6, s = slot & 63;
        const int base = page * (2 * heads * 64 * dhv);
        const int off = part == 0 ? m * d : part == 1 ? base + s * dhv : base + heads * 64 * dhv + s;
        return Row{p > T_ ? T_ : p, off};
    }
    // loads unconditionally (the V part reads an entry it ignores) so the GEMM's
    // load pipeline sees the same number of loads on every path
    __device__ Aux aux(const Row& ri, int n) const {
        const int dhv = head_dim();
        const int c = n - part * d;
        const int e = kDh ? c & (kDh - 1) : c % dhv;
        const int pi = part < 2 ? ri.p * (dhv >> 1) + (e >> 1) : 0;
        return Aux{rc[pi], rs[pi]};
    }
    // element n of a row after RoPE: q and k pairs (2i, 2i+1) turned by the
    // row/column angle of the row's position; v as is
    __device__ float value(const Aux& ax, int n, float v, float partner) const {
        if (part == 2) return v;
        const int dhv = head_dim();
        const int c = n - part * d;
        const int e = kDh ? c & (kDh - 1) : c % dhv;
        return (e & 1) ? rope_odd(partner, v, ax.cs, ax.sn) : rope_even(v, partner, ax.cs, ax.sn);
    }
    __device__ void store(const Row& ri, const Aux& ax, int m, int n, float v, float partner) const {
        const int dhv = head_dim();
        const int c = n - part * d;
        const int head = kDh ? c / kDh : c / dhv;
        const int e = c - head * dhv;
        const float out = value(ax, n, v, partner);
        const int col = part == 0 ? c : part == 1 ? head * 64 * dhv + e : head * 64 * dhv + e * 64;
        Elem<T>::store((part == 0 ? q : kv) + (ri.off + col), out);
    }
    // fp16 square tiles of BT = 64 or 128 columns (BT / 64 heads of one part)
    // are staged in LDS as fp16, tile[r * tile_ld<BT>() + c], and written from
    // there: q and K rows as 16-byte chunks (eight lanes per head row), V^T one
    // row (= cache slot) per lane, so a wavefront's store covers consecutive
    // slots of one dimension instead of 16 dimensions of 4 rows
    // (the wide kernel stages its 256 x 256 tile the same way: four heads)
    static constexpr bool stores_tile(int bt) {
        return sizeof(T) == 2 && (bt == 64 || bt == 128 || bt == 256);
    }
    template <int BT>
    __device__ int tile_ld() const { return part == 2 ? BT + 2 : BT + 8; }   // odd dwords; 16-byte rows
    // element (rl, cl) of the tile (local row and column), global column n
    __device__ void stage(uint16_t* tile, int ld, int rl, int cl, const Aux& ax, int n, float v,
                          float partner) const {
        tile[rl * ld + cl] = f32_to_f16_rne(value(ax, n, v, partner));
    }
    // a tile of TR rows and BT columns written by NT threads
    template <int BT, int TR = BT, int NT = 256>
    __device__ void store_tile(const uint16_t* tile, int n0, int m0, int M) const {
        const int t = threadIdx.x, ld = tile_ld<BT>();
        const int c0 = n0 - part * d;   // first column of the tile in its part
        const int head = c0 >> 6;
        if (part < 2) {
            constexpr int kChunks = BT / 8;   // 16-byte chunks per row
#pragma unroll
            for (int h = 0; h < TR * kChunks / NT; ++h) {
                const int qd = t + NT * h, r = qd / kChunks, col = (qd % kChunks) * 8, m = m0 + r;
                if (m < M) {
                    const Row ri = row_info(m);
                    T* dst = part == 0 ? q + ri.off + c0 + col
                                       : kv + ri.off + (head + (col >> 6)) * 64 * 64 + (col & 63);
                    *reinterpret_cast<u32x4_t*>(dst) =
                        *reinterpret_cast<const u32x4_t*>(tile + r * ld + col);
                }
            }
        } else {
            constexpr int kGroups = NT / TR;   // threads per row, each a strided set of columns
            const int r = t % TR, m = m0 + r;
            if (m < M) {
                const Row ri = row_info(m);
                T* dst = kv + ri.off + head * 64 * 64;
#pragma unroll
                for (int k = 0; k < BT / kGroups; ++k) {
                    const int e = t / BT + kGroups * k;
                    dst[(e >> 6) * 64 * 64 + (e & 63) * 64] = tile[r * ld + e];
                }
            }
        }
    }
    // The 2D RoPE factors depend only on a position's grid row (pairs below
    // dh / 4) or column (the rest) and the pair, so for a G x G grid they fit
    // in [cos, sin][row half, column half][G][dh / 4] floats, 16 G floats per
    // quarter: 8 KB at G = 32. The wide kernel gathers them from the tables
    // (entries 1 + g G and 1 + g, the same values) into LDS once per launch.
    // Returns G, or 0 when the grid does not fit (the tables are read from
    // memory then).
    static constexpr int kRopeGridMax = 32;
    __device__ int rope_grid() const {
        const int g = (int)(sqrtf((float)T_) + 0.5f);
        return kDh == 64 && g * g == T_ && g <= kRopeGridMax ? g : 0;
    }
    template <int NT>
    __device__ void load_rope(float* lds, int G) const {
        for (int k = threadIdx.x; k < 4 * G * 16; k += NT) {
            const int sc = k / (2 * G * 16), rem = k - sc * 2 * G * 16;
            const int hf = rem / (G * 16), g = (rem - hf * G * 16) >> 4, ii = k & 15;
            const int src = (hf == 0 ? 1 + g * G : 1 + g) * 32 + hf * 16 + ii;
            lds[k] = (sc == 0 ? rc : rs)[src];
        }
    }
    // The wide kernel's path: RH rows of a BT-column tile staged in LDS as fp32
    // sums before RoPE, tile[(r - rb) * ld + c] for tile rows rb .. rb + RH - 1,
    // written by NT threads; rows[i] is row_info of tile row i (the kernel
    // fetches them while the tile's main loop runs). q and K: each thread takes 8 consecutive columns
    // (four pairs of one head) of a row, fetches their four cos and four sin
    // values as two 16-byte loads, turns the pairs and stores 16 bytes. V^T:
    // each thread a row (= cache slot) and a strided set of dimensions, in
    // groups of RH threads, as many groups as a power of two that fits in NT
    // (4 groups for RH = 128 or 96, 8 for 64).
    template <int BT, int RH, int NT>
    __device__ void store_rows_f32(const float* tile, int ld, int n0, int m0, int rb, int M,
                                   const Row* rows, const float* rope, int G) const {
        const int t = threadIdx.x;
        const int c0 = n0 - part * d;
        const int head = c0 >> 6;
        if (part < 2) {
            constexpr int kChunks = BT / 8;
            static_assert(RH * kChunks % NT == 0, "q and K chunks per thread");
#pragma unroll
            for (int h = 0; h < RH * kChunks / NT; ++h) {
                const int qd = t + NT * h, r = qd / kChunks, col = (qd % kChunks) * 8;
                const int m = m0 + rb + r;
                if (m >= M) continue;
                const Row ri = rows[rb + r];
                const float4 xa = *reinterpret_cast<const float4*>(tile + r * ld + col);
                const float4 xb = *reinterpret_cast<const float4*>(tile + r * ld + col + 4);
                const int i0 = ((c0 + col) & (kDh - 1)) >> 1;   // first of four pairs
                float4 cs, sn;
                if (G) {   // the grid coordinate of the pairs' half, from LDS
                    const int hf = i0 >> 4, s1 = ri.p - 1;
                    const int g = ri.p == 0 ? 0 : hf == 0 ? s1 / G : s1 - (s1 / G) * G;
                    const float* f = rope + (hf * G + g) * 16 + (i0 & 15);
                    cs = *reinterpret_cast<const float4*>(f);
                    sn = *reinterpret_cast<const float4*>(f + 2 * G * 16);
                } else {
                    const int pi = ri.p * (kDh >> 1) + i0;
                    cs = *reinterpret_cast<const float4*>(rc + pi);
                    sn = *reinterpret_cast<const float4*>(rs + pi);
                }
                const float x[8] = {xa.x, xa.y, xa.z, xa.w, xb.x, xb.y, xb.z, xb.w};
                const float c4[4] = {cs.x, cs.y, cs.z, cs.w}, s4[4] = {sn.x, sn.y, sn.z, sn.w};
                u32x4_t out;
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    const uint32_t lo = f32_to_f16_rne(rope_even(x[2 * k], x[2 * k + 1], c4[k], s4[k]));
                    const uint32_t hi = f32_to_f16_rne(rope_odd(x[2 * k], x[2 * k + 1], c4[k], s4[k]));
                    out[k] = lo | (hi << 16);
                }
                T* dst = part == 0 ? q + ri.off + c0 + col
                                   : kv + ri.off + (head + (col >> 6)) * 64 * 64 + (col & 63);
                *reinterpret_cast<u32x4_t*>(dst) = out;
            }
        } else {
            constexpr int kGroups = NT / RH >= 8 ? 8 : NT / RH >= 4 ? 4 : NT / RH >= 2 ? 2 : 1;
            static_assert(BT % kGroups == 0, "V^T columns per thread");
            const int r = t % RH, m = m0 + rb + r;
            if (t < kGroups * RH && m < M) {
                const Row ri = rows[rb + r];
                T* dst = kv + ri.off + head * 64 * 64;
#pragma unroll 8
                for (int k = 0; k < BT / kGroups; ++k) {
                    const int e = t / RH + kGroups * k;
                    dst[(e >> 6) * 64 * 64 + (e & 63) * 64] = f32_to_f16_rne(tile[r * ld + e]);
                }
            }
        }
    }
    __device__ void operator()(int m, int n, float v, float partner) const {
        EpiQkv e = *this;
        e.part = n / d;
        const Row ri = e.row_info(m);
        e.store(ri, e.aux(ri, n), m, n, v, partner);
    }
};

// plain fp32 store of C (split-K partials of the fp32 path)
struct EpiStore {
    float* out;
    int ld;
    struct Row {};
    struct Aux {};
    __device__ void begin_tile(int) {}
    __device__ Row row_info(int) const { return Row{}; }
    __device__ Aux aux(const Row&, int) const { return Aux{}; }
    __device__ void store(const Row&, const Aux&, int m, int n, float v, float) const {
        out[(size_t)m * ld + n] = v;
    }
    __device__ void operator()(const Row& r, int m, int n, float v, float p) const {
        store(r, Aux{}, m, n, v, p);
    }
    __device__ void operator()(int m, int n, float v, float p) const { (*this)(Row{}, m, n, v, p); }
};

template <typename T>
struct EpiSwiGLU {
    T* act;
    int ld;   // f
    struct Row {};
    struct Aux {};
    __device__ void begin_tile(int) {}
    __device__ Row row_info(int) const { return Row{}; }
    __device__ Aux aux(const Row&, int) const { return Aux{}; }
    // columns 2i / 2i+1 are the gate (W1 row i) and the up projection (W3 row i).
    // With an fp16 output the logistic's reciprocal is the hardware one (1 ulp
    // in fp32, far below the output's rounding); fp32 outputs divide.
    __device__ static float swiglu(float gate, float up) {
        if constexpr (sizeof(T) == 2) {
            return gate * __builtin_amdgcn_rcpf(1.0f + __expf(-gate)) * up;
        } else {
            return gate / (1.0f + __expf(-gate)) * up;
        }
    }
    __device__ void store(const Row&, const Aux&, int m, int n, float v, float partner) const {
        if (n & 1) return;
        Elem<T>::store(act + (size_t)m * ld + (n >> 1), swiglu(v, partner));
    }
    // fp16 square tiles of BT columns give BT rows of BT / 2 outputs, staged
    // in LDS and written as 16-byte chunks per row. The 64x64 tile and the
    // wide kernel's 256x256 one use it: at 128x128 the staging measured slower
    // than storing from registers (stress rounds 48 -> 53 us per launch)
    static constexpr bool stores_tile(int bt) { return sizeof(T) == 2 && (bt == 64 || bt == 256); }
    template <int BT>
    __device__ int tile_ld() const { return BT / 2 + 8; }
    __device__ void stage(uint16_t* tile, int ld, int rl, int cl, const Aux&, int, float v,
                          float partner) const {
        if (!(cl & 1)) tile[rl * ld + (cl >> 1)] = f32_to_f16_rne(swiglu(v, partner));
    }
    // Four rows rl0 .. rl0 + 3 of column cl at once, the layout of one MFMA
    // accumulator: the lane holding the up column (odd cl) and its neighbour
    // holding the gate column trade two values each, so the gate lane computes
    // rows 0-1 and the up lane rows 2-3 and no lane computes a product it
    // throws away.
    __device__ void stage_quad(uint16_t* tile, int ld, int rl0, int cl, const f32x4_t& v) const {
        const bool up_lane = cl & 1;
        const float r0 = swap_lane_pair(up_lane ? v[0] : v[2]);
        const float r1 = swap_lane_pair(up_lane ? v[1] : v[3]);
        const float g0 = up_lane ? r0 : v[0], g1 = up_lane ? r1 : v[1];
        const float u0 = up_lane ? v[2] : r0, u1 = up_lane ? v[3] : r1;
        uint16_t* dst = tile + (rl0 + (up_lane ? 2 : 0)) * ld + (cl >> 1);
        dst[0] = f32_to_f16_rne(swiglu(g0, u0));
        dst[ld] = f32_to_f16_rne(swiglu(g1, u1));
    }
    // the same straight to the output rows m0 .. m0 + 3 (rows >= M skipped)
    __device__ void store_quad(int m0, int n, const f32x4_t& v, int M) const {
        const bool up_lane = n & 1;
        const float r0 = swap_lane_pair(up_lane ? v[0] : v[2]);
        const float r1 = swap_lane_pair(up_lane ? v[1] : v[3]);
        const float g0 = up_lane ? r0 : v[0], g1 = up_lane ? r1 : v[1];
        const float u0 = up_lane ? v[2] : r0, u1 = up_lane ? v[3] : r1;
        const int m = m0 + (up_lane ? 2 : 0);
        if (m < M) Elem<T>::store(act + (size_t)m * ld + (n >> 1), swiglu(g0, u0));
        if (m + 1 < M) Elem<T>::store(act + (size_t)(m + 1) * ld + (n >> 1), swiglu(g1, u1));
    }
    template <int BT, int TR = BT, int NT = 256>
    __device__ void store_tile(const uint16_t* tile, int n0, int m0, int M) const {
        constexpr int kChunks = BT / 16;   // 16-byte chunks per row of BT / 2 outputs
        static_assert(TR * kChunks % NT == 0, "chunks per thread");
        const int t = threadIdx.x, ldt = tile_ld<BT>();
#pragma unroll
        for (int h = 0; h < TR * kChunks / NT; ++h) {
            const int qd = t + NT * h, r = qd / kChunks, ch = qd % kChunks, m = m0 + r;
            if (m < M)
                *reinterpret_cast<u32x4_t*>(act + (size_t)m * ld + (n0 >> 1) + ch * 8) =
                    *reinterpret_cast<const u32x4_t*>(tile + r * ldt + ch * 8);
        }
    }
    __device__ void operator()(const Row& r, int m, int n, float v, float p) const {
        store(r, Aux{}, m, n, v, p);
    }
    __device__ void operator()(int m, int n, float v, float p) const { (*this)(Row{}, m, n, v, p); }
};

template <bool Bias>
struct EpiLogits {
    float* out;
    const float* bias;
    int ld;
    struct Row {};
    struct Aux { float b; };
    __device__ void begin_tile(int) {}
    __device__ Row row_info(int) const { return Row{}; }
    __device__ Aux aux(const Row&, int n) const { return Aux{Bias ? bias[n] : 0.f}; }
    __device__ void store(const Row&, const Aux& ax, int m, int n, float v, float) const {
        out[(size_t)m * ld + n] = v + ax.b;
    }
    __device__ void operator()(const Row& r, int m, int n, float v, float p) const {
        store(r, aux(r, n), m, n, v, p);
    }
    __device__ void operator()(int m, int n, float v, float p) const { (*this)(Row{}, m, n, v, p); }
};

// ---------------------------------------------------------------- fp16 MFMA
// Workgroup tile BM x BN, 4 wavefronts arranged WGM x WGN, 64-deep K steps,
// operands in LDS as rows of eight 16-byte chunks, chunk c of row r stored at
// position c ^ (r & 7) so the MFMA operand reads fall in distinct banks.
// Two ways of filling LDS, chosen per tile size:
//  * direct (kDirect): each 16-byte chunk goes from global memory straight to
//    LDS (global_load_lds_dwordx4), NS LDS stages deep, so NS-2 tiles are in
//    flight behind the one being multiplied and no registers hold them. The
//    hardware writes lane l's chunk at 16 l bytes past the wavefront's LDS
//    address, so each lane fetches the global chunk whose swizzled position
//    is l. The waits are explicit: before step kt a wavefront waits until at
//    most (NS-2) tiles' loads of its own are outstanding (loads complete in
//    issue order), then a bare s_barrier makes every wavefront's part of tile
//    kt visible. (__syncthreads would add a release fence, which waits for
//    every outstanding LDS-bound load.) A stage is refilled only after the
//    barrier that follows the step that read it.
//  * register staging: global -> registers -> LDS, double-buffered, with NS
//    register stages keeping NS-2 tiles in flight.
// Either way every step issues the same loads on every path: wait counts are
// per wavefront and in issue order, and a load skipped on some path forces a
// wait for everything. So the steady loop has no conditional loads: rows past
// M re-read row M-1 (their products land in rows that are never stored) and
// the register path's steps past the end re-read the last K tile. The
// epilogue's own inputs (row metadata, RoPE tables, bias) are fetched before
// the main loop so their latency hides behind it.
// When `part` is given the K range is cut into `splits` equal contiguous parts
// (one part with splits = 1) and each writes fp32 partial sums to `part`
// ([split][M][N]) instead of calling the epilogue; the caller's reduce kernel
// adds the parts in split order.
// An epilogue may opt out of fetching its per-element inputs before the main
// loop (static constexpr bool kLateAux = true): they are then fetched after it,
// which frees their registers during the loop at the cost of one exposed load.
template <typename E>
constexpr auto epi_prefetches_aux(int) -> decltype(E::kLateAux, bool()) { return !E::kLateAux; }
template <typename E>
constexpr bool epi_prefetches_aux(long) { return true; }
// an epilogue may stage a square fp16 tile in LDS and store it itself
// (static constexpr bool stores_tile(int tile width); stage(), store_tile())
template <typename E>
constexpr auto epi_stores_tile(int bt) -> decltype(E::stores_tile(0), bool()) {
    return E::stores_tile(bt);
}
template <typename E>
constexpr bool epi_stores_tile(long) { return false; }
// an epilogue may stage the four rows of one MFMA accumulator at once (stage_quad)
template <typename E>
constexpr auto epi_stages_quads(int) -> decltype(&E::stage_quad, bool()) { return true; }
template <typename E>
constexpr bool epi_stages_quads(long) { return false; }
// or store them from registers (store_quad)
template <typename E>
constexpr auto epi_stores_quads(int) -> decltype(&E::store_quad, bool()) { return true; }
template <typename E>
constexpr bool epi_stores_quads(long) { return false; }
// an epilogue may take the wide kernel's tile as fp32 rows (store_rows_f32)
template <typename E>
constexpr auto epi_stages_f32(int) -> decltype(&E::template store_rows_f32<256, 128, 512>, bool()) {
    return true;
}
template <typename E>
constexpr bool epi_stages_f32(long) { return false; }


// The wide kernel's tile height (32 TM rows by 256 columns, TM = 8, 6 or 4)
// and which of it and the 128 x 128 launch beside it does the work, from the
// rows present (read on the device). Each candidate costs its rounds of
// tiles times a per-round time, fitted (within 7% on average) to launches of
// the five XL products at 132-8448 rows, in hundredths of a microsecond with
// s 64-deep steps per tile: wide tiles one per CU, dealt per XCD, at
// 19.1 + 1.26 s (TM 8), 11.7 + 1.08 s (TM 6) and 7.9 + 0.84 s (TM 4);
// 128 x 128 tiles one per CU at 6.6 + 0.46 s, plus 4.4 per launch. One more
// candidate, kWideHalfTail: 256-row tiles whose last round, when at most half
// full, runs as 128-row halves (full rounds at the 256-row time, that round
// at the 128-row time). Both kernels evaluate it in the same integer
// arithmetic, so exactly one works; ties go to the wide kernel and to the
// earlier candidate in the order 256 rows, half tail, 192, 128. Returns TM
// (or kWideHalfTail), or 0 when the 128 x 128 kernel works (never with
// small = false).
constexpr int kWideHalfTail = 9;
__host__ __device__ inline long wide_cost(int tm, int M, int N, int s, int splits, int cus) {
    const int rows = 32 * (tm == kWideHalfTail ? 8 : tm);
    const long tiles = (long)((M + rows - 1) / rows) * (N / 256) * splits;
    const long slots = cus / 8, per_xcd = (tiles + 7) / 8;
    const long t8 = 1910 + 126 * s, t6 = 1170 + 108 * s, t4 = 790 + 84 * s;
    if (tm == kWideHalfTail) {
        const long full = per_xcd / slots, rest = per_xcd - full * slots;
        return rest > 0 && 2 * rest <= slots ? full * t8 + t4 : -1;   // -1: not a candidate
    }
    return (per_xcd + slots - 1) / slots * (tm == 8 ? t8 : tm == 6 ? t6 : t4);
}
__host__ __device__ inline int wide_pick(int M, int N, int K, int splits, int cus, bool small) {
    const int s = K / splits / 64;
    const long t128 = (long)((M + 127) / 128) * (N / 128) * splits;
    long best = small ? 440 + (t128 + cus - 1) / cus * (660 + 46 * s) : -1;
    int pick = 0;
    const int order[4] = {8, kWideHalfTail, 6, 4};
    for (int k = 0; k < 4; ++k) {
        const long c = wide_cost(order[k], M, N, s, splits, cus);
        if (c < 0) continue;
        if (best < 0 || (pick == 0 ? c <= best : c < best)) {
            best = c;
            pick = order[k];
        }
    }
    return pick;
}

template <int BM, int BN, int WGM, int WGN, int NS, bool kDirect, typename Epi>
__global__ __launch_bounds__(256) void k_gemm_f16(const uint16_t* __restrict__ A, int lda,
                                                  const uint16_t* __restrict__ W, float wscale,
                                                  int N, int K, const int* __restrict__ m_dev,
                                                  int m_cap, int splits, int pair_cus,
                                                  float* __restrict__ part, Epi epi) {
    constexpr int BK = 64;
    constexpr int WM = BM / WGM, WN = BN / WGN;
    constexpr int TM = WM / 16, TN = WN / 16;
    constexpr int LA = BM / 32, LB = BN / 32;   // 16-byte chunks per thread per tile
    constexpr int STAGE = (BM + BN) * BK;       // elements of one A + B stage
    // direct: NS stages; register staging: 2
    __shared__ __attribute__((aligned(1024))) uint16_t S[(kDirect ? NS : 2) * STAGE];

    const int M = m_dev ? min(*m_dev, m_cap) : m_cap;
    // launched beside the wide kernel (pair_cus = the CU count): the one of
    // the two that wide_pick picks does the work
    if (pair_cus > 0 && wide_pick(M, N, K, splits, pair_cus, true) != 0) return;
    if (M <= 0) return;
    // Persistent: the grid holds about as many workgroups as the CUs keep
    // resident, and each loops over tiles. The tiles of the rows present are
    // numbered row tile fastest, then (column tile, split); XCD x (workgroups
    // are dealt to the 8 XCDs round-robin) takes the x-th contiguous eighth,
    // all row tiles of a few (column tile, split) pairs, so it reuses weight
    // tiles in its own L2
    const int tiles_m = (M + BM - 1) / BM;
    const int total = tiles_m * (N / BN) * splits;
    const int per_xcd = (total + 7) >> 3;
    const int xcd = (int)(blockIdx.x & 7);
    const int lin_end = min((xcd + 1) * per_xcd, total);
    const int Ks = K / splits;
    const int nk = Ks / BK;
    for (int lin = xcd * per_xcd + (int)(blockIdx.x >> 3); lin < lin_end;
         lin += (int)(gridDim.x >> 3)) {
    __syncthreads();   // the previous tile is done with LDS
    const int tm = lin % tiles_m;
    const int nz = lin / tiles_m;
    const int z = nz % splits, tn = nz / splits;
    const int m0 = tm * BM, n0 = tn * BN;
    const int kbase = z * Ks;

    const int t = threadIdx.x, lane = t & 63, wv = t >> 6;
    const int wm = wv / WGN, wn = wv % WGN;

    f32x4_t acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    auto compute = [&](const uint16_t* As) {
        const uint16_t* Bs = As + BM * BK;
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
            const int ch = kk * 4 + (lane >> 4);
            f16x8_t af[TM], bfr[TN];
#pragma unroll
            for (int i = 0; i < TM; ++i) {
                const int r = wm * WM + i * 16 + (lane & 15);
                af[i] = *reinterpret_cast<const f16x8_t*>(&As[r * BK + ((ch ^ (r & 7)) << 3)]);
            }
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                const int r = wn * WN + j * 16 + (lane & 15);
                bfr[j] = *reinterpret_cast<const f16x8_t*>(&Bs[r * BK + ((ch ^ (r & 7)) << 3)]);
            }
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(af[i], bfr[j], acc[i][j],
                                                                        0, 0, 0);
        }
    };

    // epilogue inputs: row metadata first, then the first tiles, then the
    // per-element tables that depend on the row metadata
    const int col0 = n0 + wn * WN + (lane & 15);
    constexpr bool kPrefetchAux = TM * TN <= 4 && epi_prefetches_aux<Epi>(0);
    epi.begin_tile(n0);
    typename Epi::Row rinfo[TM][4];
    typename Epi::Aux aux[TM][4][TN];
    // (the split-K partial epilogue loads nothing, so this is free there)
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int v = 0; v < 4; ++v)
            rinfo[i][v] = epi.row_info(min(m0 + wm * WM + i * 16 + 4 * (lane >> 4) + v, M - 1));
    auto prefetch_aux = [&]() {
        if (kPrefetchAux) {
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int v = 0; v < 4; ++v)
#pragma unroll
                    for (int j = 0; j < TN; ++j) aux[i][v][j] = epi.aux(rinfo[i][v], col0 + j * 16);
        }
    };

    if constexpr (kDirect) {
        static_assert(NS >= 2 && NS <= 5, "direct staging depth");
        constexpr int LPT = LA + LB;   // loads per thread per tile
        // wavefront wv fills 8-row blocks wv, wv + 4, ... of each operand; lane
        // l writes row l / 8 of the block at position l % 8
        const int rr = lane >> 3;
        const int cg = (lane & 7) ^ rr;   // global chunk stored at position l % 8
        const uint16_t* asrc[LA];
        const uint16_t* bsrc[LB];
#pragma unroll
        for (int i = 0; i < LA; ++i)
            asrc[i] = A + (size_t)min(m0 + 8 * (i * 4 + wv) + rr, M - 1) * lda + kbase + cg * 8;
#pragma unroll
        for (int i = 0; i < LB; ++i)
            bsrc[i] = W + (size_t)(n0 + 8 * (i * 4 + wv) + rr) * K + kbase + cg * 8;
        auto issue = [&](int kt, int st) {
            uint16_t* sb = S + st * STAGE;
#pragma unroll
            for (int i = 0; i < LA; ++i) load_to_lds16(asrc[i] + kt * BK, sb + (i * 4 + wv) * 8 * BK);
#pragma unroll
            for (int i = 0; i < LB; ++i)
                load_to_lds16(bsrc[i] + kt * BK, sb + BM * BK + (i * 4 + wv) * 8 * BK);
        };
        // tiles 0..NS-2 into stages 0..NS-2 (a launch with fewer steps re-reads
        // its last tile, so the wait counts below still hold)
#pragma unroll
        for (int s = 0; s < NS - 1; ++s) issue(s < nk ? s : nk - 1, s);
        prefetch_aux();
        // steady steps issue one tile each, NS-1 ahead, into the stage the
        // previous step read
        const int steady = nk > NS - 1 ? nk - (NS - 1) : 0;
        int st = 0;
        for (int kt = 0; kt < steady; ++kt) {
            wait_loads<(NS - 2) * LPT>();
            lds_barrier();
            issue(kt + NS - 1, st == 0 ? NS - 1 : st - 1);
            compute(S + st * STAGE);
            st = st == NS - 1 ? 0 : st + 1;
        }
        // the last min(nk, NS-1) steps load nothing; j tiles are younger than
        // step nk-1-j's (none when the prologue re-read the last tile)
#pragma unroll
        for (int j = NS - 2; j >= 0; --j) {
            if (nk - 1 - j >= steady) {
                if (nk >= NS - 1 && j > 0) {
                    if constexpr (NS >= 5) { if (j == 3) wait_loads<3 * LPT>(); }
                    if constexpr (NS >= 4) { if (j == 2) wait_loads<2 * LPT>(); }
                    if (j == 1) wait_loads<LPT>();
                } else {
                    wait_loads<0>();
                }
                lds_barrier();
                compute(S + st * STAGE);
                st = st == NS - 1 ? 0 : st + 1;
            }
        }
    } else {
        const int lc = t & 7, lr = t >> 3;
        u32x4_t R[NS][LA + LB];
        auto gload = [&](u32x4_t* r, int kt) {
            kt = kt < nk ? kt : nk - 1;
            const int k0 = kbase + kt * BK;
#pragma unroll
            for (int i = 0; i < LA; ++i) {
                const int gm = min(m0 + lr + 32 * i, M - 1);
                r[i] = *reinterpret_cast<const u32x4_t*>(A + (size_t)gm * lda + k0 + lc * 8);
            }
#pragma unroll
            for (int i = 0; i < LB; ++i)
                r[LA + i] =
                    *reinterpret_cast<const u32x4_t*>(W + (size_t)(n0 + lr + 32 * i) * K + k0 + lc * 8);
        };
        auto sstore = [&](const u32x4_t* r, int buf) {
            uint16_t* As = S + buf * STAGE;
            uint16_t* Bs = As + BM * BK;
#pragma unroll
            for (int i = 0; i < LA; ++i) {
                const int row = lr + 32 * i;
                *reinterpret_cast<u32x4_t*>(&As[row * BK + ((lc ^ (row & 7)) << 3)]) = r[i];
            }
#pragma unroll
            for (int i = 0; i < LB; ++i) {
                const int row = lr + 32 * i;
                *reinterpret_cast<u32x4_t*>(&Bs[row * BK + ((lc ^ (row & 7)) << 3)]) = r[LA + i];
            }
        };
        // tile kt lives in register stage kt % NS
#pragma unroll
        for (int s = 0; s < NS - 1; ++s) gload(R[s], s);
        prefetch_aux();
        sstore(R[0], 0);
        __syncthreads();
        // steady state: step kt loads tile kt+NS-1 into the stage tile kt-1 left,
        // computes tile kt and moves tile kt+1 from registers to the other buffer
        const int nk_main = nk - nk % NS;
        for (int kt0 = 0; kt0 < nk_main; kt0 += NS) {
#pragma unroll
            for (int s = 0; s < NS; ++s) {
                const int kt = kt0 + s;
                gload(R[(s + NS - 1) % NS], kt + NS - 1);
                compute(S + (kt & 1) * STAGE);
                sstore(R[(s + 1) % NS], (kt + 1) & 1);
                __syncthreads();
            }
        }
        // the last nk % NS steps: their tiles were loaded by the steady loop
#pragma unroll
        for (int s = 0; s < NS - 1; ++s) {
            const int kt = nk_main + s;
            if (kt < nk) {
                compute(S + (kt & 1) * STAGE);
                if (kt + 1 < nk) sstore(R[(s + 1) % NS], (kt + 1) & 1);
                __syncthreads();
            }
        }
    }

    // the weights are held scaled by a power of two: undo it (exact)
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] *= wscale;

    // 16x16 accumulator layout: lane holds rows 4*(lane/16)+v of column lane%16
    if (part) {
        float* P = part + (size_t)z * m_cap * N;
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int row = m0 + wm * WM + i * 16 + 4 * (lane >> 4) + v;
                if (row >= M) continue;
#pragma unroll
                for (int j = 0; j < TN; ++j) P[(size_t)row * N + col0 + j * 16] = acc[i][j][v];
            }
        continue;
    }
    if (!kPrefetchAux) {
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int v = 0; v < 4; ++v)
#pragma unroll
                for (int j = 0; j < TN; ++j) aux[i][v][j] = epi.aux(rinfo[i][v], col0 + j * 16);
    }
    if constexpr (BM == BN && epi_stores_tile<Epi>(BN)) {
        __syncthreads();   // every wavefront is done with the operand stages
        uint16_t* tile = S;
        const int ld = epi.template tile_ld<BN>();
        if constexpr (epi_stages_quads<Epi>(0)) {
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    epi.stage_quad(tile, ld, wm * WM + i * 16 + 4 * (lane >> 4),
                                   wn * WN + j * 16 + (lane & 15), acc[i][j]);
        } else {
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int rl = wm * WM + i * 16 + 4 * (lane >> 4) + v;
#pragma unroll
                for (int j = 0; j < TN; ++j) {
                    const float val = acc[i][j][v];
                    const float partner = __int_as_float(__builtin_amdgcn_update_dpp(
                        0, __float_as_int(val), 0xB1, 0xF, 0xF, false));
                    epi.stage(tile, ld, rl, wn * WN + j * 16 + (lane & 15), aux[i][v][j],
                              col0 + j * 16, val, partner);
                }
            }
        }
        __syncthreads();
        epi.template store_tile<BN>(tile, n0, m0, M);
        continue;
    }
    if constexpr (epi_stores_quads<Epi>(0)) {
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j)
                epi.store_quad(m0 + wm * WM + i * 16 + 4 * (lane >> 4), col0 + j * 16, acc[i][j], M);
        continue;
    }
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int row = m0 + wm * WM + i * 16 + 4 * (lane >> 4) + v;
            const bool ok = row < M;
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                const float val = acc[i][j][v];
                // the neighbouring column's value (lane ^ 1) through a DPP quad
                // permute [1, 0, 3, 2] rather than an LDS permute
                const float partner = __int_as_float(__builtin_amdgcn_update_dpp(
                    0, __float_as_int(val), 0xB1, 0xF, 0xF, false));
                if (ok) epi.store(rinfo[i][v], aux[i][v][j], row, col0 + j * 16, val, partner);
            }
        }
    }
}

static int g_cus = 256;   // compute units of the device (gemm_setup)
// HBSJD_GEMM_TILE: "wide" (1), "wide256" / "wide192" / "wide128" (1, with the
// wide kernel's tile height fixed), "wide256h" (1, 256-row tiles with the
// half-height last round whenever it applies), "small" (-1); unset: chosen
// per launch (0)
static int g_force_tile = 0;
static int g_force_tm = 0;   // the forced height as TM (or kWideHalfTail), 0 chosen per launch

// workgroups of a 256-thread kernel one CU holds at once (looked up once per
// kernel; at least 1)
static int resident(const void* kern) {
    static std::mutex mu;
    static std::map<const void*, int> seen;
    std::lock_guard<std::mutex> lk(mu);
    auto it = seen.find(kern);
    if (it != seen.end()) return it->second;
    int n = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, kern, 256, 0) != hipSuccess || n < 1) n = 1;
    seen[kern] = n;
    return n;
}

// ---------------------------------------------------------------- wide tile
// Launches with enough rows take this kernel: 512 threads as 2 x 4
// wavefronts over a tile of 32 TM rows by 256 columns, TM = 8, 6 or 4 (256,
// 192 or 128 rows) chosen per launch by wide_pick. Each wavefront holds a
// 16 TM x 64 block of TM x 4 v_mfma_f32_16x16x32_f16 tiles whose accumulators
// live in VGPRs (two wavefronts per SIMD share the register file; a 128 x 128
// block per wavefront would fill all 256 AGPRs and the compiler then shuffles
// accumulators through VGPRs every step, measured at 0.31 of the MFMA rate
// against 0.47 for two 128 x 64 blocks). K advances 64 deep per step through
// two LDS stages (64 KB each at TM = 8) filled straight from global memory
// (rows of eight 16-byte chunks, chunk c of row r at c ^ (r & 7)): the loads
// of step k+1 are issued when step k starts. Tiles are dealt so that each
// XCD's concurrent workgroups cover about 4 row tiles x 8 column tiles, which
// its L2 serves from one read of each operand slice. Shorter tiles fill more
// CUs when a launch has few of them: 1280 output columns at 8448 rows make
// 165 tiles of 256 rows for 256 CUs but 220 of 192 rows. Every output element
// sums its K products in the same order at every height, so rows are
// bit-identical across heights and with k_gemm_f16. Split-K, wscale and the
// epilogues are those of k_gemm_f16; staged epilogues stage the whole tile in
// LDS.
constexpr int kWideN = 256, kWideK = 64;
constexpr int wide_rows(int tm) { return 32 * tm; }
constexpr int wide_stage(int tm) { return (wide_rows(tm) + kWideN) * kWideK * 2; }   // bytes
constexpr int kWideLds = wide_rows(8) * (kWideN + 8) * 2;   // the staged TM = 8 tile (> 2 stages)
// past it, the QKV epilogue's RoPE tables (EpiQkv::load_rope, G <= 32)
constexpr int kWideRopeLds = 4 * 32 * 16 * 4;
constexpr int kWideLdsTotal = kWideLds + kWideRopeLds;
static_assert(kWideLds >= 2 * wide_stage(8) && kWideLds >= wide_rows(8) / 2 * (kWideN + 4) * 4,
              "LDS of the wide kernel");
static_assert(kWideLdsTotal <= 160 * 1024, "LDS of one CU");

// one tile of k_gemm_wide at tile height 32 TM: rows m0 .. m0 + 32 TM - 1,
// columns n0 .. n0 + 255, K part z
template <int TM, typename Epi>
__device__ __forceinline__ void wide_tile(uint16_t* smem, const uint16_t* __restrict__ A, int lda,
                                          const uint16_t* __restrict__ W, float wscale, int M,
                                          int N, int K, int m_cap, int splits,
                                          float* __restrict__ part, const Epi& epi, int m0, int n0,
                                          int z, int rope_g) {
    constexpr int TN = 4, WM = TM * 16, WN = TN * 16;
    constexpr int kRows = wide_rows(TM), kStage = wide_stage(TM) / 2;   // stage in elements
    constexpr int LPW = (kRows + kWideN) / 8 / 8;   // 16-byte loads per wavefront per stage
    static_assert(TM % 2 == 0 && TM >= 4 && TM <= 8, "tile heights of 128, 192 and 256 rows");
    const int Ks = K / splits;
    const int nk = Ks / kWideK;
    const int t = threadIdx.x, lane = t & 63, wv = t >> 6;
    const int wm = wv >> 2, wn = wv & 3;
    const int lr = lane >> 3, lp = lane & 7;
    const int fr = lane & 15, fc = lane >> 4;
    // fragment offsets (elements) of the two 32-deep halves of a stage
    int aoff[2][TM], boff[2][TN];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
#pragma unroll
        for (int i = 0; i < TM; ++i) {
            const int r = wm * WM + i * 16 + fr;
            aoff[h][i] = r * kWideK + (((4 * h + fc) ^ (r & 7)) << 3);
        }
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            const int r = wn * WN + j * 16 + fr;
            boff[h][j] = kRows * kWideK + r * kWideK + (((4 * h + fc) ^ (r & 7)) << 3);
        }
    }

    const int kbase = z * Ks;

    // wavefront wv loads 8-row blocks wv, wv + 8, ... of A then of W
    const uint16_t* src[LPW];
#pragma unroll
    for (int i = 0; i < LPW; ++i) {
        const int f = wv + 8 * i;
        const int r = 8 * (f < kRows / 8 ? f : f - kRows / 8) + lr;
        const int c = (lp ^ (r & 7)) * 8;
        src[i] = f < kRows / 8 ? A + (size_t)min(m0 + r, M - 1) * lda + kbase + c
                                : W + (size_t)(n0 + r) * K + kbase + c;
    }
    auto issue = [&](int kt, int st) {
        kt = kt < nk ? kt : nk - 1;
        uint16_t* sb = smem + st * kStage;
#pragma unroll
        for (int i = 0; i < LPW; ++i) load_to_lds16(src[i] + kt * kWideK, sb + (wv + 8 * i) * 512);
    };

    f32x4_t acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    __syncthreads();   // the previous tile's epilogue is done with LDS
    issue(0, 0);
    Epi e = epi;
    e.begin_tile(n0);
    // A staged-fp32 epilogue (QKV) gets each tile row's record (position and
    // cache offset) now, into the 2 KB of LDS past its staging area: the
    // loads complete with the first stage's, which the first step waits for
    // anyway, instead of in a dependent chain after the main loop.
    typename Epi::Row* rows_lds = nullptr;
    if constexpr (epi_stages_f32<Epi>(0)) {
        static_assert(wide_rows(8) * sizeof(typename Epi::Row) <=
                          kWideLds - wide_rows(8) / 2 * (kWideN + 4) * 4,
                      "row records past the staging area");
        rows_lds = reinterpret_cast<typename Epi::Row*>(reinterpret_cast<char*>(smem) + kWideLds -
                                                        wide_rows(8) * sizeof(typename Epi::Row));
        if (t < kRows) rows_lds[t] = e.row_info(min(m0 + t, M - 1));
    }
    for (int kt = 0; kt < nk; ++kt) {
        wait_loads<0>();
        lds_barrier();
        issue(kt + 1, (kt + 1) & 1);   // the last step re-reads its own tile into the idle stage
        const uint16_t* sb = smem + (kt & 1) * kStage;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            f16x8_t a[TM], b[TN];
#pragma unroll
            for (int j = 0; j < TN; ++j) b[j] = *reinterpret_cast<const f16x8_t*>(sb + boff[h][j]);
#pragma unroll
            for (int i = 0; i < TM; ++i) a[i] = *reinterpret_cast<const f16x8_t*>(sb + aoff[h][i]);
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a[i], b[j], acc[i][j],
                                                                        0, 0, 0);
        }
        // Order of the step: the stage loads, every fragment read of both
        // halves, then the MFMAs. Right after the barrier the eight
        // wavefronts all read the same stage. Reads interleaved with the
        // MFMAs (1 per group of four) each cost a wait on the others'
        // reads, while reads issued all at once wait once (W1|W3 at 8448
        // rows on random operands: 163.6 -> 158 us; 5, 6 or 8 reads ahead
        // were slower than the 10 of the interleaved order). Masks: 0x20 VMEM
        // read, 0x100 DS read, 0x8 MFMA.
        constexpr int kReads = 2 * (TM + TN), kMfmas = 2 * TM * TN;
        __builtin_amdgcn_sched_group_barrier(0x020, LPW, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, kReads, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, kMfmas, 0);
    }
    wait_loads<0>();   // the last (redundant) stage load has landed before LDS is reused
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] *= wscale;

    const int col0 = n0 + wn * WN + (lane & 15);
    if (part) {
        float* P = part + (size_t)z * m_cap * N;
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int row = m0 + wm * WM + i * 16 + 4 * (lane >> 4) + v;
                if (row >= M) continue;
#pragma unroll
                for (int j = 0; j < TN; ++j) P[(size_t)row * N + col0 + j * 16] = acc[i][j][v];
            }
        return;
    }
    if constexpr (epi_stages_f32<Epi>(0)) {
        // two passes of 16 TM rows (the wavefronts of one wm each) in fp32
        constexpr int kLd = kWideN + 4;
        float* ft = reinterpret_cast<float*>(smem);
#pragma unroll
        for (int half = 0; half < 2; ++half) {
            __syncthreads();   // operand stages, or the previous pass, are done with LDS
            if (wm == half) {
#pragma unroll
                for (int i = 0; i < TM; ++i)
#pragma unroll
                    for (int v = 0; v < 4; ++v)
#pragma unroll
                        for (int j = 0; j < TN; ++j)
                            ft[(i * 16 + 4 * (lane >> 4) + v) * kLd + wn * WN + j * 16 + (lane & 15)] =
                                acc[i][j][v];
            }
            __syncthreads();
            e.template store_rows_f32<kWideN, kRows / 2, 512>(
                ft, kLd, n0, m0, half * (kRows / 2), M, rows_lds,
                reinterpret_cast<const float*>(reinterpret_cast<const char*>(smem) + kWideLds),
                rope_g);
        }
        return;
    } else if constexpr (epi_stores_tile<Epi>(kWideN)) {
        __syncthreads();   // every wavefront is done with the operand stages
        const int ld = e.template tile_ld<kWideN>();
        if constexpr (epi_stages_quads<Epi>(0)) {
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    e.stage_quad(smem, ld, wm * WM + i * 16 + 4 * (lane >> 4),
                                 wn * WN + j * 16 + (lane & 15), acc[i][j]);
        } else {
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int rl = wm * WM + i * 16 + 4 * (lane >> 4) + v;
                const typename Epi::Row ri = e.row_info(min(m0 + rl, M - 1));
#pragma unroll
                for (int j = 0; j < TN; ++j) {
                    const float val = acc[i][j][v];
                    const float partner = __int_as_float(__builtin_amdgcn_update_dpp(
                        0, __float_as_int(val), 0xB1, 0xF, 0xF, false));
                    e.stage(smem, ld, rl, wn * WN + j * 16 + (lane & 15),
                            e.aux(ri, col0 + j * 16), col0 + j * 16, val, partner);
                }
            }
        }
        __syncthreads();
        e.template store_tile<kWideN, kRows, 512>(smem, n0, m0, M);
        return;
    }
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int row = m0 + wm * WM + i * 16 + 4 * (lane >> 4) + v;
            const bool ok = row < M;
            const typename Epi::Row ri = e.row_info(min(row, M - 1));
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                const float val = acc[i][j][v];
                const float partner = __int_as_float(__builtin_amdgcn_update_dpp(
                    0, __float_as_int(val), 0xB1, 0xF, 0xF, false));
                if (ok) e.store(ri, e.aux(ri, col0 + j * 16), row, col0 + j * 16, val, partner);
            }
        }
}

// The persistent tile loop of k_gemm_wide at tile height 32 TM. The grid has
// at most one workgroup per CU (G of them, a multiple of 8, dealt to the XCDs
// round-robin) and each loops over tiles. The tiles of the rows present this
// launch (M <= m_cap) are numbered in groups of kGroup row tiles, column-major
// inside a group; XCD x takes the x-th contiguous eighth of that order and
// its G / 8 workgroups stride through it, so the concurrent tiles of an XCD
// share operand slices in its L2 and every XCD gets an equal share however
// few rows are present. With half_tail (TM = 8), an XCD whose last round
// would be at most half full runs that round's tiles as two 128-row halves
// each, one per workgroup: the round then costs a 128-row tile instead of a
// 256-row one.
template <int TM, typename Epi>
__device__ __forceinline__ void wide_tiles(uint16_t* smem, const uint16_t* __restrict__ A, int lda,
                                           const uint16_t* __restrict__ W, float wscale, int M,
                                           int N, int K, int m_cap, int splits,
                                           float* __restrict__ part, const Epi& epi,
                                           bool half_tail, int rope_g) {
    constexpr int kRows = wide_rows(TM), kGroup = 4;
    const int tiles_m = (M + kRows - 1) / kRows, tiles_n = N / kWideN;
    const int total = tiles_m * tiles_n * splits;
    const int per_xcd = (total + 7) >> 3;
    const int xcd = (int)(blockIdx.x & 7), slot = (int)(blockIdx.x >> 3);
    const int stride = (int)(gridDim.x >> 3);
    const int lin0 = xcd * per_xcd, lin_end = min(lin0 + per_xcd, total);
    // tile lin: K part, then groups of kGroup row tiles, column-major inside
    auto at = [&](int lin, int& m0, int& n0, int& z) {
        z = lin % splits;
        const int tl = lin / splits;
        const int grp = tl / (kGroup * tiles_n), first = grp * kGroup;
        const int gsz = min(tiles_m - first, kGroup);
        const int in = tl - grp * kGroup * tiles_n;
        m0 = (first + in % gsz) * kRows;
        n0 = (in / gsz) * kWideN;
    };
    const int count = max(lin_end - lin0, 0), full = count / stride, rest = count - full * stride;
    const bool halves = TM == 8 && half_tail && rest > 0 && 2 * rest <= stride;
    const int lin_stop = halves ? lin0 + full * stride : lin_end;
    for (int lin = lin0 + slot; lin < lin_stop; lin += stride) {
        int m0, n0, z;
        at(lin, m0, n0, z);
        wide_tile<TM>(smem, A, lda, W, wscale, M, N, K, m_cap, splits, part, epi, m0, n0, z,
                      rope_g);
    }
    if constexpr (TM == 8) {
        if (halves) {
            const int lin = lin_stop + (slot >> 1);
            if (lin < lin_end) {
                int m0, n0, z;
                at(lin, m0, n0, z);
                m0 += wide_rows(4) * (slot & 1);
                if (m0 < M)
                    wide_tile<4>(smem, A, lda, W, wscale, M, N, K, m_cap, splits, part, epi, m0, n0, z,
                                 rope_g);
            }
        }
    }
}

template <typename Epi>
__global__ __launch_bounds__(512, 1) void k_gemm_wide(const uint16_t* __restrict__ A, int lda,
                                                      const uint16_t* __restrict__ W, float wscale,
                                                      int N, int K, const int* __restrict__ m_dev,
                                                      int m_cap, int splits, int pair_cus,
                                                      int force_tm, float* __restrict__ part,
                                                      Epi epi) {
    extern __shared__ __attribute__((aligned(1024))) uint16_t smem[];
    const int M = m_dev ? min(*m_dev, m_cap) : m_cap;
    if (M <= 0) return;
    // Launched beside k_gemm_f16 (pair_cus = the CU count) it works only when
    // wide_pick picks it; alone it picks the height among its own. A nonzero
    // force_tm fixes the height (the results are the same).
    const int pick = wide_pick(M, N, K, splits, pair_cus > 0 ? pair_cus : (int)gridDim.x, pair_cus > 0);
    if (pick == 0) return;
    const int tm = force_tm ? force_tm : pick;
    // the QKV epilogue's RoPE tables, past the tile region (visible after the
    // first tile's barrier)
    int rope_g = 0;
    if constexpr (epi_stages_f32<Epi>(0)) {
        rope_g = epi.rope_grid();
        if (rope_g)
            epi.template load_rope<512>(
                reinterpret_cast<float*>(reinterpret_cast<char*>(smem) + kWideLds), rope_g);
    }
    if (tm == 4)
        wide_tiles<4>(smem, A, lda, W, wscale, M, N, K, m_cap, splits, part, epi, false, rope_g);
    else if (tm == 6)
        wide_tiles<6>(smem, A, lda, W, wscale, M, N, K, m_cap, splits, part, epi, false, rope_g);
    else
        wide_tiles<8>(smem, A, lda, W, wscale, M, N, K, m_cap, splits, part, epi,
                      tm == kWideHalfTail, rope_g);
}

// the wide kernel needs more than 64 KB of dynamic LDS: allowed once per
// epilogue type (at library set-up, before any graph capture)
template <typename Epi>
static hipError_t wide_allow_lds() {
    return hipFuncSetAttribute((const void*)k_gemm_wide<Epi>,
                               hipFuncAttributeMaxDynamicSharedMemorySize, kWideLdsTotal);
}

template <typename Epi>
static void launch_wide(const void* A, int lda, const void* W, float wscale, int N, int K,
                        const int* m_dev, int m_cap, int splits, int pair_cus, float* part,
                        const Epi& epi, hipStream_t s) {
    // sized for the capacity's tiles at the smallest height
    const int tiles = ((m_cap + wide_rows(4) - 1) / wide_rows(4)) * (N / kWideN) * splits;
    const int cap = (g_cus / 8) * 8;
    const int grid = std::max(8, std::min(cap, ((tiles + 7) / 8) * 8));
    launch(k_gemm_wide<Epi>, dim3(grid), dim3(512), (uint32_t)kWideLdsTotal, s, (const uint16_t*)A, lda,
           (const uint16_t*)W, wscale, N, K, m_dev, m_cap, splits, pair_cus, g_force_tm, part,
           epi);
}

template <int BM, int BN, int WGM, int WGN, typename Epi>
static void launch_f16(const void* A, int lda, const void* W, float wscale, int N, int K,
                       const int* m_dev, int m_cap, int splits, float* part, const Epi& epi,
                       hipStream_t s, int pair_cus = 0, int m_rows = 0) {
    if (m_cap <= 0) return;
    // sized for m_rows (the rows known on the host, at most m_cap) when given
    const int m_size = m_rows > 0 ? std::min(m_rows, m_cap) : m_cap;
    const int tiles = ((m_size + BM - 1) / BM) * (N / BN) * splits;
    // persistent grid: as many workgroups as the CUs hold at once
    auto grid_for = [&](const void* kern) {
        return std::min(((tiles + 7) / 8) * 8, std::max(8, (g_cus * resident(kern) / 8) * 8));
    };
    if constexpr (BM * BN >= 128 * 128) {
        // the large tiles have enough MFMA work per step to cover a shallow
        // register pipeline (direct staging measured no faster there)
        const int grid = grid_for((const void*)k_gemm_f16<BM, BN, WGM, WGN, 3, false, Epi>);
        launch(k_gemm_f16<BM, BN, WGM, WGN, 3, false, Epi>, dim3(grid), dim3(256), 0, s,
               (const uint16_t*)A, lda, (const uint16_t*)W, wscale, N, K, m_dev, m_cap, splits,
               pair_cus, part, epi);
    } else if (tiles <= 512) {
        // direct staging, 4 stages (64 KB of LDS): two workgroups per CU hold
        // the whole launch
        const int grid = grid_for((const void*)k_gemm_f16<BM, BN, WGM, WGN, 4, true, Epi>);
        launch(k_gemm_f16<BM, BN, WGM, WGN, 4, true, Epi>, dim3(grid), dim3(256), 0, s,
               (const uint16_t*)A, lda, (const uint16_t*)W, wscale, N, K, m_dev, m_cap, splits,
               pair_cus, part, epi);
    } else {
        // more tiles than two per CU: 3 stages (48 KB), three workgroups per CU
        const int grid = grid_for((const void*)k_gemm_f16<BM, BN, WGM, WGN, 3, true, Epi>);
        launch(k_gemm_f16<BM, BN, WGM, WGN, 3, true, Epi>, dim3(grid), dim3(256), 0, s,
               (const uint16_t*)A, lda, (const uint16_t*)W, wscale, N, K, m_dev, m_cap, splits,
               pair_cus, part, epi);
    }
}

// tile choice by the launch's row cap (the same for Full and Compact rounds):
// large tiles once there are enough of them to fill the 256 CUs twice over
// Launches whose rows are only known on the device (m_dev) and that could
// fill the wide kernel take both it and the smaller-tile kernel; each reads
// the row count and wide_pick tells which one works. (A persistent launch
// that finds no work costs a few microseconds; a wide-tile launch sized for
// the capacity would cost its idle workgroups' dispatch, about as much as
// the work of a full launch.) With a host-side bound on the rows
// (gemm_row_bound) only the kernel wide_pick picks for the bound is launched.
constexpr int kWideMin = 96;   // capacity in 256 x 256 tiles below which it is not tried

static thread_local int g_row_bound = -1;
static thread_local std::vector<GemmPlan>* g_plan_log = nullptr;
void gemm_row_bound(int rows) { g_row_bound = rows; }
void gemm_plan_log(std::vector<GemmPlan>* log) { g_plan_log = log; }

// rows known on the host, exactly (no device count) or as an upper bound
// (0: neither)
static int host_rows(bool m_dev, int m_cap, int row_bound) {
    return !m_dev ? m_cap : row_bound >= 0 ? std::max(1, std::min(row_bound, m_cap)) : 0;
}

// the kernels of a product of N x K weights over up to m_cap rows (m_dev: the
// row count is read on the device), under the calling thread's row bound
static int plan_kernels(int N, int K, bool m_dev, int m_cap, int splits, bool wide_ok,
                        int row_bound) {
    const long t256 = (long)((m_cap + 255) / 256) * (N / 256) * splits;
    const bool fit = wide_ok && N % 256 == 0 && (K / splits) % kWideK == 0;
    const int m_host = host_rows(m_dev, m_cap, row_bound);
    // the smaller tiles: 64 x 64 while the CUs hold all of them at once (3 per
    // CU; 4 stages deep up to 512 tiles, as launch_f16 sizes them), else
    // 128 x 128. Measured with the partial-sum store at 132-5478 rows of the
    // XL products: once 64 x 64 needs a second round, 128 x 128 took at most
    // as long (W2 at 2640 rows 51 -> 40 us), except QKV at 1188 rows (23 ->
    // 26 us), where the wide kernel works.
    const int m_sel = m_host > 0 ? m_host : m_cap;
    const long t64 = (long)((m_sel + 63) / 64) * (N / 64) * splits;
    const int small = N % 128 == 0 && t64 > 3L * g_cus ? kGemm128 : t64 <= 512 ? kGemm64 | kGemmDeep : kGemm64;
    if (g_force_tile != 0)   // HBSJD_GEMM_TILE: one kernel for every launch (results are the same)
        return g_force_tile > 0 && fit ? kGemmWide : small;
    const bool wide = fit && t256 >= kWideMin;
    // with host rows, the kernel wide_pick picks for that many rows, alone
    if (m_host > 0) return wide && wide_pick(m_host, N, K, splits, g_cus, true) != 0 ? kGemmWide : small;
    return wide ? small | kGemmPair : small;
}

int gemm_plan(const GemmPlan& p, int row_bound) {
    return plan_kernels(p.N, p.K, true, p.m_cap, p.splits, p.wide_ok, row_bound);
}

template <typename Epi>
static void dispatch_f16(const void* A, int lda, const void* W, float wscale, int N, int K,
                         const int* m_dev, int m_cap, int splits, float* part, const Epi& epi,
                         hipStream_t s, bool wide_ok = true) {
    const int k = plan_kernels(N, K, m_dev != nullptr, m_cap, splits, wide_ok, g_row_bound);
    if (g_plan_log && m_dev) g_plan_log->push_back(GemmPlan{N, K, m_cap, splits, wide_ok, k});
    // a pair: both kernels, each reads the row count and wide_pick tells which one works
    const int pair = k & kGemmPair ? g_cus : 0;
    if (k & (kGemmWide | kGemmPair))
        launch_wide(A, lda, W, wscale, N, K, m_dev, m_cap, splits, pair, part, epi, s);
    const int m_rows = host_rows(m_dev != nullptr, m_cap, g_row_bound);
    if ((k & 3) == kGemm128)
        launch_f16<128, 128, 2, 2>(A, lda, W, wscale, N, K, m_dev, m_cap, splits, part, epi, s, pair,
                                   m_rows);
    else if ((k & 3) == kGemm64)
        launch_f16<64, 64, 2, 2>(A, lda, W, wscale, N, K, m_dev, m_cap, splits, part, epi, s, pair,
                                 m_rows);
}

// ---------------------------------------------------------------- fp32

template <typename Epi>
__global__ __launch_bounds__(256) void k_gemm_f32(const float* __restrict__ A, int lda,
                                                  const float* __restrict__ W, int N, int K,
                                                  const int* __restrict__ m_dev, int m_cap,
                                                  Epi epi) {
    __shared__ float As[16][68];
    __shared__ float Bs[16][68];
    const int M = m_dev ? min(*m_dev, m_cap) : m_cap;
    const int m0 = blockIdx.y * 64, n0 = blockIdx.x * 64;
    if (m0 >= M) return;
    const int t = threadIdx.x, ty = t >> 4, tx = t & 15;
    float acc[4][4] = {};
    for (int k0 = 0; k0 < K; k0 += 16) {
        {
            const int r = t >> 2, kk = (t & 3) * 4;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int gm = m0 + r, gk = k0 + kk + i, gn = n0 + r;
                As[kk + i][r] = (gm < M && gk < K) ? A[(size_t)gm * lda + gk] : 0.f;
                Bs[kk + i][r] = (gn < N && gk < K) ? W[(size_t)gn * K + gk] : 0.f;
            }
        }
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < 16; ++kk) {
            float a[4], b[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) a[i] = As[kk][ty * 4 + i];
#pragma unroll
            for (int j = 0; j < 4; ++j) b[j] = Bs[kk][tx * 4 + j];
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
        }
        __syncthreads();
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int row = m0 + ty * 4 + i;
        if (row >= M) continue;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int col = n0 + tx * 4 + j;
            if (col < N) epi(row, col, acc[i][j], acc[i][j ^ 1]);
        }
    }
}

template <typename Epi>
static void launch_f32(const void* A, int lda, const void* W, int N, int K, const int* m_dev,
                       int m_cap, const Epi& epi, hipStream_t s) {
    if (m_cap <= 0) return;
    dim3 grid((N + 63) / 64, (m_cap + 63) / 64);
    launch(k_gemm_f32<Epi>, grid, dim3(256), 0, s, (const float*)A, lda,
                       (const float*)W, N, K, m_dev, m_cap, epi);
}

// ---------------------------------------------------------------- entry points

int split_for(int m_cap, int N, int K) {
    // enough (tile, split) pairs for about two 64x64 workgroups per CU, at most
    // four parts, each a whole number of 64-deep steps
    const long tiles = (long)((m_cap + 63) / 64) * (N / 64);
    int want = (int)((512 + tiles - 1) / tiles);
    want = want < 1 ? 1 : (want > 4 ? 4 : want);
    const int steps = K / 64;
    int sp = 1;
    for (int c = 1; c <= want; ++c)
        if (steps % c == 0) sp = c;
    return sp;
}

void gemm_qkv(bool f16, const void* A, int lda, const void* W, float wscale, int N, int K,
              const int* m_dev, int m_cap, const QkvArgs& e, hipStream_t s) {
    if (f16) {
        EpiQkv<uint16_t> epi{(uint16_t*)e.q, (uint16_t*)e.kv, e.pos, e.kvslot, e.rope_cos,
                             e.rope_sin, e.d, e.heads, e.head_dim, e.T};
        // a 256-column tile must lie inside one of q, k and v
        dispatch_f16(A, lda, W, wscale, N, K, m_dev, m_cap, 1, nullptr, epi, s, e.d % 256 == 0);
    } else {
        EpiQkv<float> epi{(float*)e.q, (float*)e.kv, e.pos, e.kvslot, e.rope_cos, e.rope_sin,
                          e.d, e.heads, e.head_dim, e.T};
        launch_f32(A, lda, W, N, K, m_dev, m_cap, epi, s);
    }
}

template <int Tag>   // 0 the O projection, 1 W2 (distinct kernel names in traces)
struct PartialTag {};

// the split-K partial sums are written by the kernel itself; no epilogue
template <int Tag>
struct EpiNone {
    struct Row {};
    struct Aux {};
    __device__ void begin_tile(int) {}
    __device__ Row row_info(int) const { return Row{}; }
    __device__ Aux aux(const Row&, int) const { return Aux{}; }
    __device__ void store(const Row&, const Aux&, int, int, float, float) const {}
    PartialTag<Tag> tag;
};

template <int Tag>
static void partial_tag(bool f16, const void* A, int lda, const void* W, float wscale, int N,
                        int K, const int* m_dev, int m_cap, int splits, float* part,
                        hipStream_t s) {
    if (f16) {
        dispatch_f16(A, lda, W, wscale, N, K, m_dev, m_cap, splits, part, EpiNone<Tag>{}, s);
    } else {
        launch_f32(A, lda, W, N, K, m_dev, m_cap, EpiStore{part, N}, s);
    }
}

// The residual stream h += A W^T (rows below the count), when the product has
// one K part: each element is added to h once by the tile that owns it, the
// same single fp32 addition the norm kernel makes with a one-part sum.
template <int Tag>
struct EpiResidual {
    float* h;
    int ld;
    struct Row {};
    struct Aux {};
    __device__ void begin_tile(int) {}
    __device__ Row row_info(int) const { return Row{}; }
    __device__ Aux aux(const Row&, int) const { return Aux{}; }
    __device__ void store(const Row&, const Aux&, int m, int n, float v, float) const {
        float* p = h + (size_t)m * ld + n;
        *p = *p + v;
    }
    // The wide kernel stages its tile in LDS as fp32 rows and each thread
    // updates 16 bytes of a row at a time (the same additions).
    __device__ int rope_grid() const { return 0; }
    template <int NT>
    __device__ void load_rope(float*, int) const {}
    template <int BT, int RH, int NT>
    __device__ void store_rows_f32(const float* tile, int ld_t, int n0, int m0, int rb, int M,
                                   const Row*, const float*, int) const {
        constexpr int kQuads = BT / 4;
        static_assert(RH * kQuads % NT == 0, "quads per thread");
        const int t = threadIdx.x;
#pragma unroll
        for (int k = 0; k < RH * kQuads / NT; ++k) {
            const int qd = t + NT * k, r = qd / kQuads, c = (qd % kQuads) * 4;
            const int m = m0 + rb + r;
            if (m >= M) continue;
            float4* p = reinterpret_cast<float4*>(h + (size_t)m * ld + n0 + c);
            const float4 v = *reinterpret_cast<const float4*>(tile + r * ld_t + c);
            const float4 x = *p;
            *p = make_float4(x.x + v.x, x.y + v.y, x.z + v.z, x.w + v.w);
        }
    }
    PartialTag<Tag> tag;
};

void gemm_residual(int tag, const void* A, int lda, const void* W, float wscale, int N, int K,
                   const int* m_dev, int m_cap, float* h, hipStream_t s) {
    if (tag == 0)
        dispatch_f16(A, lda, W, wscale, N, K, m_dev, m_cap, 1, nullptr, EpiResidual<0>{h, N}, s);
    else
        dispatch_f16(A, lda, W, wscale, N, K, m_dev, m_cap, 1, nullptr, EpiResidual<1>{h, N}, s);
}

void gemm_partial(bool f16, int tag, const void* A, int lda, const void* W, float wscale, int N,
                  int K, const int* m_dev, int m_cap, int splits, float* part, hipStream_t s) {
    if (tag == 0)
        partial_tag<0>(f16, A, lda, W, wscale, N, K, m_dev, m_cap, splits, part, s);
    else
        partial_tag<1>(f16, A, lda, W, wscale, N, K, m_dev, m_cap, splits, part, s);
}

void gemm_swiglu(bool f16, const void* A, int lda, const void* W, float wscale, int N, int K,
                 const int* m_dev, int m_cap, void* act, hipStream_t s) {
    if (f16) {
        EpiSwiGLU<uint16_t> epi{(uint16_t*)act, N / 2};
        dispatch_f16(A, lda, W, wscale, N, K, m_dev, m_cap, 1, nullptr, epi, s);
    } else {
        EpiSwiGLU<float> epi{(float*)act, N / 2};
        launch_f32(A, lda, W, N, K, m_dev, m_cap, epi, s);
    }
}

void gemm_logits(bool f16, const void* A, int lda, const void* W, float wscale, int N, int K,
                 const int* m_dev, int m_cap, float* out, const float* bias, hipStream_t s) {
    if (bias) {
        EpiLogits<true> epi{out, bias, N};
        if (f16)
            dispatch_f16(A, lda, W, wscale, N, K, m_dev, m_cap, 1, nullptr, epi, s);
        else
            launch_f32(A, lda, W, N, K, m_dev, m_cap, epi, s);
    } else {
        EpiLogits<false> epi{out, nullptr, N};
        if (f16)
            dispatch_f16(A, lda, W, wscale, N, K, m_dev, m_cap, 1, nullptr, epi, s);
        else
            launch_f32(A, lda, W, N, K, m_dev, m_cap, epi, s);
    }
}

static_assert(epi_stages_f32<EpiQkv<uint16_t>>(0) && !epi_stages_f32<EpiSwiGLU<uint16_t>>(0),
              "the wide kernel stages QKV tiles as fp32 rows");

hipError_t gemm_setup() {
    const char* f = std::getenv("HBSJD_GEMM_TILE");
    g_force_tile = 0;
    g_force_tm = 0;
    if (f) {
        const struct { const char* name; int tile, tm; } opts[] = {
            {"wide", 1, 0},      {"wide256", 1, 8}, {"wide256h", 1, kWideHalfTail},
            {"wide192", 1, 6},   {"wide128", 1, 4}, {"small", -1, 0}};
        for (const auto& o : opts)
            if (std::strcmp(f, o.name) == 0) {
                g_force_tile = o.tile;
                g_force_tm = o.tm;
            }
    }
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) == hipSuccess &&
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess &&
        cus >= 8)
        g_cus = cus;
    const hipError_t e[] = {wide_allow_lds<EpiQkv<uint16_t>>(), wide_allow_lds<EpiSwiGLU<uint16_t>>(),
                            wide_allow_lds<EpiLogits<true>>(), wide_allow_lds<EpiLogits<false>>(),
                            wide_allow_lds<EpiNone<0>>(), wide_allow_lds<EpiNone<1>>(),
                            wide_allow_lds<EpiResidual<0>>(), wide_allow_lds<EpiResidual<1>>()};
    for (hipError_t x : e)
        if (x != hipSuccess) return x;
    return hipSuccess;
}

// ---------------------------------------------------------------- MFMA calibration
// Every wavefront issues iters x 8 independent v_mfma_f32_16x16x32_f16 back to
// back with no memory traffic: a kernel whose matrix cores are busy for its
// whole run, against which the MFMA counters and the sustained rate are read.
// The sums reach memory only if they equal a value they cannot take.
__global__ __launch_bounds__(256) void k_mfma_probe(int iters, float* __restrict__ sink) {
    const float x = (float)(threadIdx.x & 7) * 0.125f;
    f16x8_t a, b;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        a[e] = (_Float16)(x + 0.25f * e);
        b[e] = (_Float16)(0.5f - x);
    }
    f32x4_t acc[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) acc[k] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    for (int i = 0; i < iters; ++i) {
#pragma unroll
        for (int k = 0; k < 8; ++k) acc[k] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, acc[k], 0, 0, 0);
    }
    float t = 0.f;
#pragma unroll
    for (int k = 0; k < 8; ++k) t += acc[k][0] + acc[k][1] + acc[k][2] + acc[k][3];
    if (t == -1234567.f) sink[threadIdx.x] = t;
}

void mfma_probe(int workgroups, int iters, float* sink, hipStream_t s) {
    launch(k_mfma_probe, dim3(workgroups), dim3(256), 0, s, iters, sink);
}

}  // namespace hbsjd
