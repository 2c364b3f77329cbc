// Teacher scoring after the rollout: the per-position bidirectional KL between
// the student's and the teacher's next-token distributions on the completed
// sequences, and its mean over the generated positions (Sec. 3.1, Eq. 3).
#include <hip/hip_runtime.h>

#include "common.h"
#include "launch.h"

namespace hbsjd {
namespace {

typedef float f32x4_t __attribute__((ext_vector_type(4)));

// One 256-thread block per pair of logits rows. Thread t keeps float4 chunks
// t, t + 256, ... of both rows in registers (NV chunks per row), so the rows
// are read from HBM once and the three passes below run on registers:
//   1. the two maxima;
//   2. the two normalisers Z_s = sum exp(ls - m_s), Z_t likewise;
//   3. sum_v (p_v - q_v) (ls_v - lt_v) / 2.
// The last sum is KL(p||q)/2 + KL(q||p)/2: log p - log q = (ls - lt) minus a
// constant, and the constant drops out because sum_v (p_v - q_v) = 0. Summing
// differences of probabilities (rather than two expectations of ls - lt)
// keeps the result accurate when the two distributions are close.
template <int NV>
__global__ __launch_bounds__(256) void k_bikl(const float* __restrict__ ls,
                                             const float* __restrict__ lt, int V, int rows,
                                             const int32_t* __restrict__ out_idx,
                                             float* __restrict__ out) {
    __shared__ float red[4];
    const int r = blockIdx.x;
    if (r >= rows) return;
    const int t = threadIdx.x;
    const int nv4 = V >> 2;
    const f32x4_t* s4 = reinterpret_cast<const f32x4_t*>(ls + (size_t)r * V);
    const f32x4_t* t4 = reinterpret_cast<const f32x4_t*>(lt + (size_t)r * V);
    f32x4_t a[NV], b[NV];
#pragma unroll
    for (int j = 0; j < NV; ++j) {
        // clamped index: every load is issued unconditionally, the entries
        // past V are masked out below
        const int i = min(t + 256 * j, nv4 - 1);
        a[j] = s4[i];
        b[j] = t4[i];
    }
    float ms = -INFINITY, mt = -INFINITY;
#pragma unroll
    for (int j = 0; j < NV; ++j) {
        const bool ok = t + 256 * j < nv4;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            ms = fmaxf(ms, ok ? a[j][c] : -INFINITY);
            mt = fmaxf(mt, ok ? b[j][c] : -INFINITY);
        }
    }
    auto fmax2 = [](float x, float y) { return fmaxf(x, y); };
    auto add2 = [](float x, float y) { return x + y; };
    ms = block_reduce(ms, red, fmax2);
    mt = block_reduce(mt, red, fmax2);
    float zs = 0.f, zt = 0.f;
#pragma unroll
    for (int j = 0; j < NV; ++j) {
        const bool ok = t + 256 * j < nv4;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            zs += ok ? __expf(a[j][c] - ms) : 0.f;
            zt += ok ? __expf(b[j][c] - mt) : 0.f;
        }
    }
    zs = block_reduce(zs, red, add2);
    zt = block_reduce(zt, red, add2);
    const float is = 1.f / zs, it = 1.f / zt;
    float acc = 0.f;
#pragma unroll
    for (int j = 0; j < NV; ++j) {
        const bool ok = t + 256 * j < nv4;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            // both products rounded on their own (no fused multiply-add), so
            // swapping the two models negates dp exactly
            const float dp = __fmul_rn(__expf(a[j][c] - ms), is) - __fmul_rn(__expf(b[j][c] - mt), it);
            acc += ok ? dp * (a[j][c] - b[j][c]) : 0.f;
        }
    }
    acc = block_reduce(acc, red, add2);
    if (t == 0) out[out_idx ? out_idx[r] : r] = 0.5f * acc;
}

// One 256-thread block per image: mean of its generated positions' values.
__global__ __launch_bounds__(256) void k_bikl_mean(const float* __restrict__ per,
                                                  const int32_t* __restrict__ k, int T,
                                                  float* __restrict__ loss) {
    __shared__ float red[4];
    const int b = blockIdx.x, t = threadIdx.x;
    const int k0 = k[b];
    float s = 0.f;
    for (int i = k0 + t; i < T; i += 256) s += per[(size_t)b * T + i];
    s = block_reduce(s, red, [](float x, float y) { return x + y; });
    if (t == 0) loss[b] = k0 < T ? s / (float)(T - k0) : 0.f;
}

}  // namespace

void bikl_rows(const float* ls, const float* lt, int rows, int V, const int32_t* out_idx,
               float* out, hipStream_t s) {
    if (rows <= 0) return;
    const int nv4 = V / 4;
    const int per = (nv4 + 255) / 256;
    const dim3 grid(rows), block(256);
    if (per <= 1)
        launch(k_bikl<1>, grid, block, 0, s, ls, lt, V, rows, out_idx, out);
    else if (per <= 2)
        launch(k_bikl<2>, grid, block, 0, s, ls, lt, V, rows, out_idx, out);
    else if (per <= 4)
        launch(k_bikl<4>, grid, block, 0, s, ls, lt, V, rows, out_idx, out);
    else if (per <= 8)
        launch(k_bikl<8>, grid, block, 0, s, ls, lt, V, rows, out_idx, out);
    else
        launch(k_bikl<16>, grid, block, 0, s, ls, lt, V, rows, out_idx, out);
}

void bikl_mean(const float* per, const int32_t* k, int B, int T, float* loss, hipStream_t s) {
    if (B <= 0) return;
    launch(k_bikl_mean, dim3(B), dim3(256), 0, s, per, k, T, loss);
}

}  // namespace hbsjd
