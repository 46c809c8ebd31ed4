// Shared device helpers for the gfx950 kernels: storage types, 16-byte
// vector I/O, wave64 reductions and the counter-based dropout generator.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dm {

typedef _Float16 half_t;
typedef __bf16 bf16_t;
typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// ------------------------------------------------------------ conversions
__device__ __forceinline__ float to_f(float x) { return x; }
__device__ __forceinline__ float to_f(half_t x) { return (float)x; }
__device__ __forceinline__ float to_f(bf16_t x) { return (float)x; }

template <typename T> __device__ __forceinline__ T from_f(float x);
template <> __device__ __forceinline__ float from_f<float>(float x) { return x; }
template <> __device__ __forceinline__ half_t from_f<half_t>(float x) { return (half_t)x; }
template <> __device__ __forceinline__ bf16_t from_f<bf16_t>(float x) { return (bf16_t)x; }

// --------------------------------------------- 8-element vector load/store
// Every activation row has a multiple of 8 elements and 16-byte aligned
// bases, so 8 consecutive elements are one (half/bf16) or two (float)
// 16-byte transactions.
template <typename T> struct V8;

template <> struct V8<half_t> {
    // 8 elements already loaded as 16 raw bytes
    __device__ __forceinline__ static void unpack(u32x4 r, float v[8]) {
        half8 h = __builtin_bit_cast(half8, r);
#pragma unroll
        for (int i = 0; i < 8; ++i) v[i] = (float)h[i];
    }
    __device__ __forceinline__ static void load(const half_t* p, float v[8]) {
        unpack(*reinterpret_cast<const u32x4*>(p), v);
    }
    __device__ __forceinline__ static u32x4 pack(const float v[8]) {
        half8 h;
#pragma unroll
        for (int i = 0; i < 8; ++i) h[i] = (half_t)v[i];
        return __builtin_bit_cast(u32x4, h);
    }
    __device__ __forceinline__ static void store(half_t* p, const float v[8]) {
        *reinterpret_cast<u32x4*>(p) = pack(v);
    }
};

template <> struct V8<bf16_t> {
    // 8 elements already loaded as 16 raw bytes; bf16 -> fp32 is a 16-bit
    // shift of the bit pattern
    __device__ __forceinline__ static void unpack(u32x4 r, float v[8]) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            v[2 * i] = __builtin_bit_cast(float, r[i] << 16);
            v[2 * i + 1] = __builtin_bit_cast(float, r[i] & 0xFFFF0000u);
        }
    }
    __device__ __forceinline__ static void load(const bf16_t* p, float v[8]) {
        unpack(*reinterpret_cast<const u32x4*>(p), v);
    }
    __device__ __forceinline__ static u32x4 pack(const float v[8]) {
        bf16x8 h;
#pragma unroll
        for (int i = 0; i < 8; ++i) h[i] = (bf16_t)v[i];
        return __builtin_bit_cast(u32x4, h);
    }
    __device__ __forceinline__ static void store(bf16_t* p, const float v[8]) {
        *reinterpret_cast<u32x4*>(p) = pack(v);
    }
};

template <> struct V8<float> {
    __device__ __forceinline__ static void load(const float* p, float v[8]) {
        floatx4 a = *reinterpret_cast<const floatx4*>(p);
        floatx4 b = *reinterpret_cast<const floatx4*>(p + 4);
#pragma unroll
        for (int i = 0; i < 4; ++i) { v[i] = a[i]; v[4 + i] = b[i]; }
    }
    __device__ __forceinline__ static void store(float* p, const float v[8]) {
        floatx4 a, b;
#pragma unroll
        for (int i = 0; i < 4; ++i) { a[i] = v[i]; b[i] = v[4 + i]; }
        *reinterpret_cast<floatx4*>(p) = a;
        *reinterpret_cast<floatx4*>(p + 4) = b;
    }
};

// ------------------------------------------------------ wave64 reductions
// Reduction over `width` consecutive lanes (a power of two <= 64); every
// lane of the group receives the result.  Within a row of 16 lanes the
// partners come from DPP operand permutations, which cost one VALU
// instruction per step (a lane shuffle through the LDS unit costs about
// seven, with an LDS round trip): quad_perm [1,0,3,2] and [2,3,0,1] pair
// lanes 1 and 2 apart, then row_half_mirror (lane i <-> 7 - i within 8) and
// row_mirror (i <-> 15 - i within 16) join the halves that already hold
// their partial results.  Across rows: one shuffle for 32 lanes; for the
// whole wave the four row results are read into scalar registers, so the
// result is wave-uniform.
namespace dpp {
constexpr int QUAD_XOR1 = 0xB1, QUAD_XOR2 = 0x4E, ROW_HALF_MIRROR = 0x141, ROW_MIRROR = 0x140;
template <int CTRL>
__device__ __forceinline__ float perm(float v) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xF, 0xF, false));
}
}  // namespace dpp

template <int WIDTH, typename Op>
__device__ __forceinline__ float group_reduce(float v, Op op) {
    static_assert(WIDTH >= 1 && WIDTH <= 64 && (WIDTH & (WIDTH - 1)) == 0, "group width");
    if constexpr (WIDTH >= 2) v = op(v, dpp::perm<dpp::QUAD_XOR1>(v));
    if constexpr (WIDTH >= 4) v = op(v, dpp::perm<dpp::QUAD_XOR2>(v));
    if constexpr (WIDTH >= 8) v = op(v, dpp::perm<dpp::ROW_HALF_MIRROR>(v));
    if constexpr (WIDTH >= 16) v = op(v, dpp::perm<dpp::ROW_MIRROR>(v));
    if constexpr (WIDTH == 32) v = op(v, __shfl_xor(v, 16, 64));
    if constexpr (WIDTH == 64) {
        const float r0 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 0));
        const float r1 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 16));
        const float r2 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 32));
        const float r3 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 48));
        v = op(op(r0, r1), op(r2, r3));
    }
    return v;
}
// e^(x - m) for the softmax rows, as 2^(x log2(e) - m log2(e)): one fma and
// one v_exp_f32 per element (the subtraction folds into the fma; results
// below 2^-126 flush to zero, far under the storage types' resolution).
struct ExpShift {
    float ml;
    __device__ __forceinline__ explicit ExpShift(float m) : ml(m * 1.4426950408889634f) {}
    __device__ __forceinline__ float operator()(float x) const {
        return __builtin_amdgcn_exp2f(fmaf(x, 1.4426950408889634f, -ml));
    }
};

template <int WIDTH>
__device__ __forceinline__ float group_sum(float v) {
    return group_reduce<WIDTH>(v, [](float a, float b) { return a + b; });
}
template <int WIDTH>
__device__ __forceinline__ float group_max(float v) {
    return group_reduce<WIDTH>(v, [](float a, float b) { return fmaxf(a, b); });
}

// ------------------------------------------------- counter-based dropout
// Philox4x32 with 10 rounds (Salmon, Moraes, Dror, Shaw, SC'11): the round
// multiplies counter words 0 and 2 by two constants and mixes the high
// product halves with words 1 and 3 and the round key; the key is bumped by
// two Weyl constants between rounds.  Each 32x32 -> 64-bit product is one
// v_mad_u64_u32 (both halves at once) and each three-way mix one
// v_bitop3_b32, about half the instructions of separate high / low
// multiplies and two-input xors; the generator is ALU-bound in the fused
// kernels that draw masks.
// a ^ b ^ k with k wave-uniform (the round keys derive from kernel
// arguments only), taken from a scalar register: gfx950's three-input
// bitwise operation with truth table 0x96 (odd parity of the three bits)
__device__ __forceinline__ uint32_t xor3(uint32_t a, uint32_t b, uint32_t k) {
    uint32_t r;
    asm("v_bitop3_b32 %0, %1, %2, %3 bitop3:0x96" : "=v"(r) : "v"(a), "v"(b), "s"(k));
    return r;
}

struct Philox {
    static constexpr uint32_t M0 = 0xD2511F53u, M1 = 0xCD9E8D57u;
    static constexpr uint32_t W0 = 0x9E3779B9u, W1 = 0xBB67AE85u;
    __device__ __forceinline__ static u32x4 gen(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3,
                                                uint32_t k0, uint32_t k1) {
#pragma unroll
        for (int r = 0; r < 10; ++r) {
            const uint64_t p0 = (uint64_t)c0 * M0, p1 = (uint64_t)c2 * M1;
            const uint32_t n0 = xor3((uint32_t)(p1 >> 32), c1, k0), n2 = xor3((uint32_t)(p0 >> 32), c3, k1);
            c0 = n0; c1 = (uint32_t)p1; c2 = n2; c3 = (uint32_t)p0;
            k0 += W0; k1 += W1;
        }
        u32x4 o; o[0] = c0; o[1] = c1; o[2] = c2; o[3] = c3;
        return o;
    }
};

// Dropout parameters as the kernels see them.  The mask of logical element
// e is word (e & 3) of Philox(counter = (lo(e>>2), hi(e>>2), site, layer),
// key = (lo(seed), hi(seed))); keep iff word < thr.  thr == 2^32 keeps all.
struct DropParams {
    uint64_t seed;
    uint64_t thr;      // floor((1-p) * 2^32), in [0, 2^32]
    uint32_t site, layer;
    float scale;       // 1/(1-p)
    int enabled;       // p > 0
};

// Multiplies 8 values of logical elements e0..e0+7 (e0 % 8 == 0) by the
// dropout factor.
__device__ __forceinline__ void dropout8(const DropParams& d, uint64_t e0, float v[8]) {
    if (!d.enabled) return;
    uint64_t blk = e0 >> 2;
    uint32_t k0 = (uint32_t)d.seed, k1 = (uint32_t)(d.seed >> 32);
    u32x4 a = Philox::gen((uint32_t)blk, (uint32_t)(blk >> 32), d.site, d.layer, k0, k1);
    blk += 1;
    u32x4 b = Philox::gen((uint32_t)blk, (uint32_t)(blk >> 32), d.site, d.layer, k0, k1);
    // enabled means p > 0, so thr < 2^32 fits 32 bits
    const uint32_t thr = (uint32_t)d.thr;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        v[i] = a[i] < thr ? v[i] * d.scale : 0.0f;
        v[4 + i] = b[i] < thr ? v[4 + i] * d.scale : 0.0f;
    }
}

// Keep bits of logical elements e0..e0+7 as 0/1 bytes.
__device__ __forceinline__ void keep8(const DropParams& d, uint64_t e0, uint8_t out[8]) {
    if (!d.enabled) {
#pragma unroll
        for (int i = 0; i < 8; ++i) out[i] = 1;
        return;
    }
    uint64_t blk = e0 >> 2;
    uint32_t k0 = (uint32_t)d.seed, k1 = (uint32_t)(d.seed >> 32);
    u32x4 a = Philox::gen((uint32_t)blk, (uint32_t)(blk >> 32), d.site, d.layer, k0, k1);
    blk += 1;
    u32x4 b = Philox::gen((uint32_t)blk, (uint32_t)(blk >> 32), d.site, d.layer, k0, k1);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        out[i] = a[i] < (uint32_t)d.thr;
        out[4 + i] = b[i] < (uint32_t)d.thr;
    }
}

// ----------------------------------------------------------- activations
enum Act { ACT_GELU = 0, ACT_RELU = 1 };

// erf(x) for x >= 0 and e = exp(-x^2), by the rational approximation of
// Abramowitz & Stegun, Handbook of Mathematical Functions, 7.1.26:
// erf(x) = 1 - t (a1 + t (a2 + t (a3 + t (a4 + t a5)))) e, t = 1 / (1 + p x),
// absolute error <= 1.5e-7.  The exponential is the one the GELU density
// needs anyway (exp(-u^2 / 2) with x = u / sqrt 2), so GELU and its
// derivative cost one exp and one reciprocal.
__device__ __forceinline__ float erf_pos(float x, float e) {
    const float t = __builtin_amdgcn_rcpf(fmaf(0.3275911f, x, 1.0f));
    const float poly =
        t * fmaf(t, fmaf(t, fmaf(t, fmaf(t, 1.061405429f, -1.453152027f), 1.421413741f), -0.284496736f),
                 0.254829592f);
    return fmaf(-poly, e, 1.0f);
}

// GELU (exact erf form): Phi(u) = (1 + erf(u / sqrt 2)) / 2
__device__ __forceinline__ float gelu_cdf(float u, float& e) {
    const float x = u * 0.70710678118654752f;
    e = __expf(-x * x);
    const float ea = erf_pos(fabsf(x), e);
    return 0.5f + 0.5f * (x < 0.0f ? -ea : ea);
}

__device__ __forceinline__ float act_fwd(float u, int act) {
    if (act == ACT_RELU) return fmaxf(u, 0.0f);
    float e;
    return u * gelu_cdf(u, e);
}
// d/du of the activation: GELU' = Phi(u) + u * phi(u), phi(u) = exp(-u^2/2) / sqrt(2 pi)
__device__ __forceinline__ float act_grad(float u, int act) {
    if (act == ACT_RELU) return u > 0.0f ? 1.0f : 0.0f;
    float e;
    const float cdf = gelu_cdf(u, e);
    return fmaf(u * 0.39894228040143268f, e, cdf);
}

}  // namespace dm
