// Shared device helpers of the HIP library (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace hbsjd {

// ------------------------------------------------------------ constants

constexpr int kPage = 64;       // KV slots per page; also the attention key tile
constexpr int kChunk = 64;      // vocabulary sums run sequentially inside 64-entry chunks
constexpr int kMaxVocab = 16384;
constexpr int kMaxChunks = kMaxVocab / kChunk;

// per-round device bookkeeping written by the round set-up kernel (int32 slots)
enum MetaSlot : int {
    kMetaRows = 0,     // rows in the verifier forward (all CFG branches)
    kMetaOutRows = 1,  // distribution rows (one per image and window row)
    kMetaImgs = 2,     // images physically processed this round
    kMetaSegs = 3,     // attention segments (one per sequence processed)
    kMetaActive = 4,   // A: images that still have tokens to generate
    kMetaMode = 5,     // 0 Full, 1 Compact
    kMetaRound = 6,    // index of the round in progress
    kMetaError = 7,    // sticky device error bits
    kMetaGamma = 8,    // Full/Compact threshold of AUTO rounds
    kMetaExec = 9,     // 0 AUTO, 1 FULL, 2 COMPACT
    kMetaSeedLo = 10,  // Philox key, low and high words
    kMetaSeedHi = 11,
    kMetaCount = 16,
};

enum DeviceError : int {
    kErrNanLogit = 1,
    kErrZeroProposal = 2,
    kErrBadToken = 4,
    kErrRoundOverflow = 8,
};

// ------------------------------------------------------------ 16-bit numbers
// A bf16 model's weights are rounded to bf16 (nearest-even) on load. The MFMA
// operands, the activations between kernels and the KV cache are fp16: the
// same operand width and matrix-core rate as bf16, with three more mantissa
// bits. Each weight matrix is held as fp16 times a power of two (its scale), so
// every bf16 weight of the matrix down to 2^-31 of its largest magnitude is
// represented exactly; the GEMMs multiply their fp32 sums by the inverse scale.

__host__ __device__ inline uint16_t f32_to_bf16(float f) {
    uint32_t u;
    __builtin_memcpy(&u, &f, 4);
    if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x007FFFFFu)) return (uint16_t)((u >> 16) | 0x40);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

__host__ __device__ inline float bf16_to_f32(uint16_t h) {
    uint32_t u = (uint32_t)h << 16;
    float f;
    __builtin_memcpy(&f, &u, 4);
    return f;
}

// fp32 -> fp16 bits, round to nearest even, for the host's weight conversion
// (finite inputs whose magnitude is below 65520; larger ones give infinity)
inline uint16_t f32_to_f16_bits_host(float f) {
    uint32_t u;
    __builtin_memcpy(&u, &f, 4);
    const uint16_t sign = (uint16_t)((u >> 16) & 0x8000u);
    const int e = (int)((u >> 23) & 0xFF) - 127;
    uint32_t m = u & 0x7FFFFFu;
    if (e > 15) return sign | 0x7C00u;
    if (e >= -14) {   // normal: keep 10 of the 23 mantissa bits
        uint32_t h = ((uint32_t)(e + 15) << 10) | (m >> 13);
        const uint32_t rest = m & 0x1FFFu;
        if (rest > 0x1000u || (rest == 0x1000u && (h & 1u))) ++h;   // may carry into the exponent
        return sign | (uint16_t)h;
    }
    if (e < -25) return sign;   // below half the smallest subnormal
    // subnormal: value = m' * 2^-24 with m' = (1.m) * 2^(e + 24)
    m |= 0x800000u;
    const int shift = -e - 1;   // 14 .. 24: bits of the 24-bit significand dropped
    uint32_t h = m >> shift;
    const uint32_t rest = m & ((1u << shift) - 1u), half = 1u << (shift - 1);
    if (rest > half || (rest == half && (h & 1u))) ++h;
    return sign | (uint16_t)h;
}

// device conversions use the hardware converts (round to nearest even)
__device__ inline uint16_t f32_to_f16_rne(float f) { return __builtin_bit_cast(uint16_t, (_Float16)f); }
__device__ inline float f16_to_f32(uint16_t h) { return (float)__builtin_bit_cast(_Float16, h); }

template <typename T> struct Elem;
template <> struct Elem<float> {
    __device__ static float load(const float* p) { return *p; }
    __device__ static void store(float* p, float v) { *p = v; }
};
template <> struct Elem<uint16_t> {
    __device__ static float load(const uint16_t* p) { return f16_to_f32(*p); }
    __device__ static void store(uint16_t* p, float v) { *p = f32_to_f16_rne(v); }
};

// ------------------------------------------------------------ Philox4x32-10

// Counter-based generator of Salmon, Moraes, Dror and Shaw (SC'11): ten
// rounds of the two-multiply bijection, the key bumped by the Weyl constants
// between rounds.
struct U4 { uint32_t x, y, z, w; };

__host__ __device__ inline U4 philox4x32_10(uint64_t seed, uint32_t c0, uint32_t c1,
                                            uint32_t c2, uint32_t c3) {
    uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        const uint64_t m0 = (uint64_t)0xD2511F53u * c0;
        const uint64_t m1 = (uint64_t)0xCD9E8D57u * c2;
        const uint32_t n0 = (uint32_t)(m1 >> 32) ^ c1 ^ k0;
        const uint32_t n1 = (uint32_t)m1;
        const uint32_t n2 = (uint32_t)(m0 >> 32) ^ c3 ^ k1;
        const uint32_t n3 = (uint32_t)m0;
        c0 = n0; c1 = n1; c2 = n2; c3 = n3;
        k0 += 0x9E3779B9u;
        k1 += 0xBB67AE85u;
    }
    return U4{c0, c1, c2, c3};
}

// uniform on [0, 1 - 2^-24] from the 24 high bits
__host__ __device__ inline float unit_float(uint32_t x) {
    return (float)(x >> 8) * (1.0f / 16777216.0f);
}

__device__ inline uint64_t meta_seed(const int32_t* meta) {
    return ((uint64_t)(uint32_t)meta[kMetaSeedHi] << 32) | (uint32_t)meta[kMetaSeedLo];
}

// the three uniforms of image b at sequence position t: draft, accept, resample
struct Uniforms { float draft, acc, res; };
__device__ __forceinline__ Uniforms uniforms_at(uint64_t seed, int b, int t) {
    const U4 o = philox4x32_10(seed, (uint32_t)b, (uint32_t)t, 0u, 0u);
    return Uniforms{unit_float(o.x), unit_float(o.y), unit_float(o.z)};
}

// ------------------------------------------------------------ reductions

__device__ inline float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}
__device__ inline float wave_max(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
    return v;
}
__device__ inline float wave_min(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fminf(v, __shfl_xor(v, o, 64));
    return v;
}
__device__ inline int wave_min_int(int v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = min(v, __shfl_xor(v, o, 64));
    return v;
}
__device__ inline int wave_max_int(int v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = max(v, __shfl_xor(v, o, 64));
    return v;
}
__device__ inline int wave_sum_int(int v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

// block-wide reductions for 256-thread blocks (fixed tree order)
template <typename F>
__device__ inline float block_reduce(float v, float* red, F op) {
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = op(v, __shfl_xor(v, o, 64));
    __syncthreads();
    if (lane == 0) red[wid] = v;
    __syncthreads();
    float r = op(op(red[0], red[1]), op(red[2], red[3]));
    __syncthreads();
    return r;
}

// one 16-byte chunk per lane from global memory to LDS: lane l's chunk lands
// at lds + 16 l (lds is the same for the whole wavefront)
__device__ __forceinline__ void load_to_lds16(const void* g, void* lds) {
    __builtin_amdgcn_global_load_lds(g, (__attribute__((address_space(3))) void*)lds, 16, 0, 0);
}
// workgroup barrier alone; the memory clobber keeps the compiler from moving
// LDS accesses across it
__device__ __forceinline__ void lds_barrier() { asm volatile("s_barrier" ::: "memory"); }
// wait until at most N vector memory loads of this wavefront are outstanding
template <int N>
__device__ __forceinline__ void wait_loads() {
    static_assert(N >= 0 && N < 64, "vmcnt is 6 bits");
    // s_waitcnt fields: vmcnt[3:0], expcnt[6:4], lgkmcnt[11:8], vmcnt[5:4] at [15:14]
    __builtin_amdgcn_s_waitcnt((N & 15) | (0x7 << 4) | (0xF << 8) | ((N >> 4) << 14));
}

}  // namespace hbsjd
