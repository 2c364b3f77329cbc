// Dense contractions of the verifier forward: QKV, O, W1|W3 and W2 projections
// and the lm_head, each C = A . W^T with the neighbouring elementwise work
// fused into the epilogue (2D RoPE and the paged KV append after QKV, the
// residual add after O and W2, SwiGLU after W1|W3, bias after the lm_head).
//
// bf16 path: 256-thread workgroups, 2x2 wavefronts, LDS-staged double-buffered
// 64-deep K tiles with an XOR swizzle, v_mfma_f32_16x16x32_bf16 with fp32
// accumulation. Every output element sums its K range in the same order no
// matter how many rows the launch has or where the row sits, so a row's result
// does not depend on the rest of the batch.
// fp32 path: a plain LDS-tiled FMA kernel for the exact-parity mode.
#include "common.h"
#include "launch.h"

namespace hbsjd {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(4))) float f32x4_t;

// ---------------------------------------------------------------- epilogues
// operator()(row, col, value, value of column col ^ 1 in the same row)

template <typename T>
struct EpiQkv {
    T* q;
    T* kv;
    const int32_t* pos;
    const int32_t* kvslot;
    const float* rc;
    const float* rs;
    int d, heads, dh, T_;
    __device__ void operator()(int m, int n, float v, float partner) const {
        const int part = n / d;
        const int c = n - part * d;
        const int head = c / dh, e = c - head * dh;
        float out = v;
        if (part < 2) {
            int p = pos[m];
            p = p > T_ ? T_ : p;
            const int pi = p * (dh >> 1) + (e >> 1);
            const float cs = rc[pi], sn = rs[pi];
            // adjacent pair (2i, 2i+1) turned by the row/column angle of position p
            out = (e & 1) ? (partner * sn + v * cs) : (v * cs - partner * sn);
        }
        if (part == 0) {
            Elem<T>::store(q + (size_t)m * d + c, out);
            return;
        }
        const int slot = kvslot[m];
        const int page = slot >> 6, s = slot & 63;
        const size_t base = (size_t)page * (2 * heads * 64 * dh);
        if (part == 1)
            Elem<T>::store(kv + base + (size_t)head * 64 * dh + (size_t)s * dh + e, out);
        else
            Elem<T>::store(kv + base + (size_t)(heads + head) * 64 * dh + (size_t)e * 64 + s, out);
    }
};

template <int Tag>   // 0 after the O projection, 1 after W2 (distinct kernel names)
struct EpiResidual {
    float* h;
    int ld;
    __device__ void operator()(int m, int n, float v, float) const {
        float* p = h + (size_t)m * ld + n;
        *p = *p + v;
    }
};

template <typename T>
struct EpiSwiGLU {
    T* act;
    int ld;   // f
    // columns 2i / 2i+1 are the gate (W1 row i) and the up projection (W3 row i)
    __device__ void operator()(int m, int n, float v, float partner) const {
        if (n & 1) return;
        const float silu = v / (1.0f + __expf(-v));
        Elem<T>::store(act + (size_t)m * ld + (n >> 1), silu * partner);
    }
};

struct EpiLogits {
    float* out;
    const float* bias;
    int ld;
    __device__ void operator()(int m, int n, float v, float) const {
        out[(size_t)m * ld + n] = bias ? v + bias[n] : v;
    }
};

// ---------------------------------------------------------------- bf16 MFMA

template <int BM, int BN, typename Epi>
__global__ __launch_bounds__(256) void k_gemm_bf16(const uint16_t* __restrict__ A, int lda,
                                                   const uint16_t* __restrict__ W, int N, int K,
                                                   const int* __restrict__ m_dev, int m_cap,
                                                   Epi epi) {
    constexpr int BK = 64;
    constexpr int WM = BM / 2, WN = BN / 2;
    constexpr int TM = WM / 16, TN = WN / 16;
    constexpr int LA = BM / 32, LB = BN / 32;   // 16-byte chunks per thread per tile
    __shared__ __attribute__((aligned(16))) uint16_t As[2][BM * BK];
    __shared__ __attribute__((aligned(16))) uint16_t Bs[2][BN * BK];

    const int M = m_dev ? min(*m_dev, m_cap) : m_cap;
    const int tiles_m = (m_cap + BM - 1) / BM;
    const int total = tiles_m * (N / BN);
    const int per_xcd = (total + 7) >> 3;
    // workgroups are dealt to the 8 XCDs round-robin; give each XCD a contiguous
    // range of tiles (all M tiles of a few N tiles) so it reuses weight tiles in its L2
    const int lin = (int)(blockIdx.x & 7) * per_xcd + (int)(blockIdx.x >> 3);
    if (lin >= total) return;
    const int tn = lin / tiles_m, tm = lin - tn * tiles_m;
    const int m0 = tm * BM, n0 = tn * BN;
    if (m0 >= M) return;

    const int t = threadIdx.x, lane = t & 63, wv = t >> 6;
    const int wm = wv >> 1, wn = wv & 1;
    const int lc = t & 7, lr = t >> 3;

    uint4 ra[LA], rb[LB];
    auto gload = [&](int k0) {
#pragma unroll
        for (int i = 0; i < LA; ++i) {
            const int r = lr + 32 * i;
            const int gm = m0 + r;
            if (gm < M)
                ra[i] = *reinterpret_cast<const uint4*>(A + (size_t)gm * lda + k0 + lc * 8);
            else
                ra[i] = make_uint4(0, 0, 0, 0);
        }
#pragma unroll
        for (int i = 0; i < LB; ++i) {
            const int r = lr + 32 * i;
            rb[i] = *reinterpret_cast<const uint4*>(W + (size_t)(n0 + r) * K + k0 + lc * 8);
        }
    };
    auto sstore = [&](int buf) {
#pragma unroll
        for (int i = 0; i < LA; ++i) {
            const int r = lr + 32 * i;
            *reinterpret_cast<uint4*>(&As[buf][r * BK + ((lc ^ (r & 7)) << 3)]) = ra[i];
        }
#pragma unroll
        for (int i = 0; i < LB; ++i) {
            const int r = lr + 32 * i;
            *reinterpret_cast<uint4*>(&Bs[buf][r * BK + ((lc ^ (r & 7)) << 3)]) = rb[i];
        }
    };

    f32x4_t acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    const int nk = K / BK;
    gload(0);
    sstore(0);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
        const int buf = kt & 1;
        if (kt + 1 < nk) gload((kt + 1) * BK);
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
            const int ch = kk * 4 + (lane >> 4);
            bf16x8_t af[TM], bfr[TN];
#pragma unroll
            for (int i = 0; i < TM; ++i) {
                const int r = wm * WM + i * 16 + (lane & 15);
                af[i] = *reinterpret_cast<const bf16x8_t*>(&As[buf][r * BK + ((ch ^ (r & 7)) << 3)]);
            }
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                const int r = wn * WN + j * 16 + (lane & 15);
                bfr[j] = *reinterpret_cast<const bf16x8_t*>(&Bs[buf][r * BK + ((ch ^ (r & 7)) << 3)]);
            }
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bfr[j], acc[i][j],
                                                                        0, 0, 0);
        }
        if (kt + 1 < nk) sstore(buf ^ 1);
        __syncthreads();
    }

    // 16x16 accumulator layout: lane holds rows 4*(lane/16)+v of column lane%16
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const float val = acc[i][j][v];
                const float partner = __shfl_xor(val, 1, 64);
                const int row = m0 + wm * WM + i * 16 + 4 * (lane >> 4) + v;
                const int col = n0 + wn * WN + j * 16 + (lane & 15);
                if (row < M) epi(row, col, val, partner);
            }
}

template <int BM, int BN, typename Epi>
static void launch_bf16(const void* A, int lda, const void* W, int N, int K, const int* m_dev,
                        int m_cap, const Epi& epi, hipStream_t s) {
    if (m_cap <= 0) return;
    const int tiles = ((m_cap + BM - 1) / BM) * (N / BN);
    const int grid = ((tiles + 7) / 8) * 8;
    launch(k_gemm_bf16<BM, BN, Epi>, dim3(grid), dim3(256), 0, s,
                       (const uint16_t*)A, lda, (const uint16_t*)W, N, K, m_dev, m_cap, epi);
}

// tile choice: enough workgroups to cover the 256 CUs at the launch's row cap
template <typename Epi>
static void dispatch_bf16(const void* A, int lda, const void* W, int N, int K, const int* m_dev,
                          int m_cap, const Epi& epi, hipStream_t s) {
    const long big = (long)((m_cap + 127) / 128) * (N / 128);
    if (N % 128 == 0 && big >= 512)
        launch_bf16<128, 128>(A, lda, W, N, K, m_dev, m_cap, epi, s);
    else if (N % 128 == 0 && (long)((m_cap + 63) / 64) * (N / 128) >= 256)
        launch_bf16<64, 128>(A, lda, W, N, K, m_dev, m_cap, epi, s);
    else
        launch_bf16<64, 64>(A, lda, W, N, K, m_dev, m_cap, epi, s);
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

void gemm_qkv(bool bf16, const void* A, int lda, const void* W, int N, int K, const int* m_dev,
              int m_cap, const QkvArgs& e, hipStream_t s) {
    if (bf16) {
        EpiQkv<uint16_t> epi{(uint16_t*)e.q, (uint16_t*)e.kv, e.pos, e.kvslot, e.rope_cos,
                             e.rope_sin, e.d, e.heads, e.head_dim, e.T};
        dispatch_bf16(A, lda, W, N, K, m_dev, m_cap, epi, s);
    } else {
        EpiQkv<float> epi{(float*)e.q, (float*)e.kv, e.pos, e.kvslot, e.rope_cos, e.rope_sin,
                          e.d, e.heads, e.head_dim, e.T};
        launch_f32(A, lda, W, N, K, m_dev, m_cap, epi, s);
    }
}

template <int Tag>
static void residual_tag(bool bf16, const void* A, int lda, const void* W, int N, int K,
                         const int* m_dev, int m_cap, float* h, hipStream_t s) {
    EpiResidual<Tag> epi{h, N};
    if (bf16)
        dispatch_bf16(A, lda, W, N, K, m_dev, m_cap, epi, s);
    else
        launch_f32(A, lda, W, N, K, m_dev, m_cap, epi, s);
}

void gemm_residual(bool bf16, int tag, const void* A, int lda, const void* W, int N, int K,
                   const int* m_dev, int m_cap, float* h, hipStream_t s) {
    if (tag == 0)
        residual_tag<0>(bf16, A, lda, W, N, K, m_dev, m_cap, h, s);
    else
        residual_tag<1>(bf16, A, lda, W, N, K, m_dev, m_cap, h, s);
}

void gemm_swiglu(bool bf16, const void* A, int lda, const void* W, int N, int K,
                 const int* m_dev, int m_cap, void* act, hipStream_t s) {
    if (bf16) {
        EpiSwiGLU<uint16_t> epi{(uint16_t*)act, N / 2};
        dispatch_bf16(A, lda, W, N, K, m_dev, m_cap, epi, s);
    } else {
        EpiSwiGLU<float> epi{(float*)act, N / 2};
        launch_f32(A, lda, W, N, K, m_dev, m_cap, epi, s);
    }
}

void gemm_logits(bool bf16, const void* A, int lda, const void* W, int N, int K,
                 const int* m_dev, int m_cap, float* out, const float* bias, hipStream_t s) {
    EpiLogits epi{out, bias, N};
    if (bf16)
        dispatch_bf16(A, lda, W, N, K, m_dev, m_cap, epi, s);
    else
        launch_f32(A, lda, W, N, K, m_dev, m_cap, epi, s);
}

}  // namespace hbsjd
