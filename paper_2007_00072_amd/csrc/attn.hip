// Attention-score kernels that never write the score tensor to HBM.
//
// Forward (Table 3 rows QK^T and scaled softmax + dropout, the paper's
// contraction followed by its `sm` operator): each block computes the
// scaled scores beta = s * Q K^T of 32 query rows against all K keys of one
// (b, h) on 32x32x16 MFMAs, rounds them to the storage type into LDS (the
// value the two-kernel path writes to HBM), and then runs the row softmax
// + dropout of those rows from LDS, writing the probabilities P and
// alpha = dropout(P).
//
// Backward (Table 3 rows Gamma dX1 and `bs`): each block computes
// d(alpha) = d(gamma) V^T for 32 query rows, rounds it into LDS the same
// way, reads P and regenerates the dropout mask, and writes
// d(beta) = s * P * (dP - sum_k dP P), dP = dropout(d(alpha)).
//
// Either kernel saves one write and one read of a B*H*J*K tensor against
// the separate contraction and row-operator launches.
//
// The MFMA operands come straight from global memory: lane l of a 32x32x16
// step holds row l % 32 of its operand at 8 contraction indices, and since
// the sum over the contraction index may run in any order, the lanes of
// half-wave hh take indices [hh D/2, (hh + 1) D/2) in D/16 steps of 8, i.e.
// each lane reads D/2 contiguous elements of its row.
#include <math.h>

#include "internal.hpp"

namespace dm {
namespace {

constexpr int NTA = 512;  // threads per block: 8 waves

template <typename T> struct AMfma;
template <> struct AMfma<half_t> {
    __device__ __forceinline__ static floatx16 run(u32x4 a, u32x4 b, floatx16 c) {
        return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(half8, a), __builtin_bit_cast(half8, b), c,
                                                      0, 0, 0);
    }
};
template <> struct AMfma<bf16_t> {
    __device__ __forceinline__ static floatx16 run(u32x4 a, u32x4 b, floatx16 c) {
        return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b),
                                                       c, 0, 0, 0);
    }
};

// Operand rows: element (z = b*H + h, row r, contraction index d) at
// ptr + b*outer + h*inner + r*ld + d.
struct AttnOp {
    const void* ptr;
    int64_t outer, inner, ld;
};

struct AttnArgs {
    AttnOp a;            // query-side rows (Q, or d(gamma) token-major)
    AttnOp b;            // key-side rows (K, or V)
    int B, H, J, K, D;   // D: contraction length (P or W)
    float out_scale;     // applied to the contraction before rounding (s forward, 1 backward)
    float sm_scale;      // backward: s multiplying d(beta)
    DropParams dp;       // attention-probability dropout (site 0)
    const void* prob;    // backward: P
    void* out0;          // forward: P        backward: d(beta)
    void* out1;          // forward: alpha
};

template <typename T, int LPR, int NV, int DK, bool BWD>
__global__ __launch_bounds__(NTA) void attn_fused_k(AttnArgs g) {
    extern __shared__ __attribute__((aligned(16))) unsigned char smem_raw[];
    T* S = reinterpret_cast<T*>(smem_raw);
    const int K = g.K, J = g.J, pitch = K + 16;  // 4 rows apart = 32 banks mod 64: the half-waves' writes do not collide
    const int z = blockIdx.y, j0 = blockIdx.x * 32;
    const int b = z / g.H, h = z - b * g.H;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, c = lane & 31, hh = lane >> 5;

    // ---- contraction: S[32][K] = out_scale * A_rows . B_rows^T
    {
        const int jr = min(j0 + c, J - 1);
        const T* arow = reinterpret_cast<const T*>(g.a.ptr) + b * g.a.outer + h * g.a.inner + jr * g.a.ld +
                        hh * (g.D / 2);
        u32x4 af[DK];
#pragma unroll
        for (int s = 0; s < DK; ++s) af[s] = *reinterpret_cast<const u32x4*>(arow + 8 * s);
        const T* bbase = reinterpret_cast<const T*>(g.b.ptr) + b * g.b.outer + h * g.b.inner + hh * (g.D / 2);
        for (int cb = wave; cb < K / 32; cb += NTA / 64) {
            const T* brow = bbase + (int64_t)(cb * 32 + c) * g.b.ld;
            u32x4 bf[DK];
#pragma unroll
            for (int s = 0; s < DK; ++s) bf[s] = *reinterpret_cast<const u32x4*>(brow + 8 * s);
            floatx16 acc;
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[r] = 0.f;
#pragma unroll
            for (int s = 0; s < DK; ++s) acc = AMfma<T>::run(af[s], bf[s], acc);
#pragma unroll
            for (int r = 0; r < 16; ++r)
                S[(8 * (r >> 2) + 4 * hh + (r & 3)) * pitch + cb * 32 + c] = from_f<T>(acc[r] * g.out_scale);
        }
    }
    __syncthreads();

    // ---- row phase: one lane group of LPR lanes per row, NV 8-element vectors per lane
    constexpr int RPW = 64 / LPR;
    const int gi = lane / LPR, gl = lane % LPR;
    const int nr = min(32, J - j0);
    for (int rb = 0; rb < 32; rb += (NTA / 64) * RPW) {
        const int lr = rb + wave * RPW + gi;
        const bool active = lr < nr;
        const int j = j0 + lr;
        const int64_t base = ((int64_t)z * J + j) * K;              // row of P / alpha / d(beta)
        const int64_t ebase = (((int64_t)h * g.B + b) * J + j) * K;  // dropout logical index (h, b, j, k)
        float v[NV][8];
        if constexpr (!BWD) {
            float mx = -INFINITY;
#pragma unroll
            for (int i = 0; i < NV; ++i) {
                const int col = (gl + i * LPR) * 8;
                if (active && col < K) {
                    V8<T>::unpack(*reinterpret_cast<const u32x4*>(S + lr * pitch + col), v[i]);
#pragma unroll
                    for (int q = 0; q < 8; ++q) mx = fmaxf(mx, v[i][q]);
                } else {
#pragma unroll
                    for (int q = 0; q < 8; ++q) v[i][q] = -INFINITY;
                }
            }
            mx = group_max<LPR>(mx);
            float sum = 0.f;
#pragma unroll
            for (int i = 0; i < NV; ++i)
#pragma unroll
                for (int q = 0; q < 8; ++q) { v[i][q] = __expf(v[i][q] - mx); sum += v[i][q]; }
            sum = group_sum<LPR>(sum);
            if (!active) continue;
            const float rinv = 1.0f / sum;
#pragma unroll
            for (int i = 0; i < NV; ++i) {
                const int col = (gl + i * LPR) * 8;
                if (col < K) {
#pragma unroll
                    for (int q = 0; q < 8; ++q) v[i][q] *= rinv;
                    V8<T>::store(reinterpret_cast<T*>(g.out0) + base + col, v[i]);
                    dropout8(g.dp, (uint64_t)(ebase + col), v[i]);
                    V8<T>::store(reinterpret_cast<T*>(g.out1) + base + col, v[i]);
                }
            }
        } else {
            float p[NV][8];
            float dot = 0.f;
#pragma unroll
            for (int i = 0; i < NV; ++i) {
                const int col = (gl + i * LPR) * 8;
                if (active && col < K) {
                    V8<T>::load(reinterpret_cast<const T*>(g.prob) + base + col, p[i]);
                    V8<T>::unpack(*reinterpret_cast<const u32x4*>(S + lr * pitch + col), v[i]);
                    dropout8(g.dp, (uint64_t)(ebase + col), v[i]);
#pragma unroll
                    for (int q = 0; q < 8; ++q) dot += v[i][q] * p[i][q];
                } else {
#pragma unroll
                    for (int q = 0; q < 8; ++q) { v[i][q] = 0.f; p[i][q] = 0.f; }
                }
            }
            dot = group_sum<LPR>(dot);
            if (!active) continue;
#pragma unroll
            for (int i = 0; i < NV; ++i) {
                const int col = (gl + i * LPR) * 8;
                if (col < K) {
                    float o[8];
#pragma unroll
                    for (int q = 0; q < 8; ++q) o[q] = g.sm_scale * p[i][q] * (v[i][q] - dot);
                    V8<T>::store(reinterpret_cast<T*>(g.out0) + base + col, o);
                }
            }
        }
    }
}

template <typename T, bool BWD>
void attn_fused_t(const AttnArgs& g, hipStream_t st) {
    const dim3 grid((g.J + 31) / 32, g.B * g.H);
    const size_t lds = (size_t)32 * (g.K + 16) * sizeof(T);
    const int len = g.K;
#define L(LPR, NV)                                                                                                \
    {                                                                                                             \
        switch (g.D / 16) {                                                                                       \
            case 1: hipLaunchKernelGGL((attn_fused_k<T, LPR, NV, 1, BWD>), grid, dim3(NTA), lds, st, g); break; \
            case 2: hipLaunchKernelGGL((attn_fused_k<T, LPR, NV, 2, BWD>), grid, dim3(NTA), lds, st, g); break; \
            case 3: hipLaunchKernelGGL((attn_fused_k<T, LPR, NV, 3, BWD>), grid, dim3(NTA), lds, st, g); break; \
            case 4: hipLaunchKernelGGL((attn_fused_k<T, LPR, NV, 4, BWD>), grid, dim3(NTA), lds, st, g); break; \
            case 6: hipLaunchKernelGGL((attn_fused_k<T, LPR, NV, 6, BWD>), grid, dim3(NTA), lds, st, g); break; \
            default: hipLaunchKernelGGL((attn_fused_k<T, LPR, NV, 8, BWD>), grid, dim3(NTA), lds, st, g); break; \
        }                                                                                                         \
    }
    if (len <= 32) { L(4, 1) }
    else if (len <= 64) { L(8, 1) }
    else if (len <= 128) { L(16, 1) }
    else if (len <= 256) { L(32, 1) }
    else if (len <= 512) { L(64, 1) }
    else { L(64, 2) }
#undef L
}

AttnOp attn_op(const void* p, int64_t outer, int64_t inner, int64_t ld) {
    AttnOp o;
    o.ptr = p; o.outer = outer; o.inner = inner; o.ld = ld;
    return o;
}

}  // namespace

bool attn_fused_ok(int dtype, int K, int D) {
    // the score tile (32 rows of K + 16 elements) stays within 64 KB of LDS
    return (dtype == DM_F16 || dtype == DM_BF16) && K % 32 == 0 && K <= 960 &&
           (D == 16 || D == 32 || D == 48 || D == 64 || D == 96 || D == 128);
}

void run_attn_scores_fwd(int dtype, int B, int H, int J, int K, int D, float scaler, const void* q, int64_t q_outer,
                         int64_t q_inner, int64_t q_ld, const void* k, int64_t k_outer, int64_t k_inner, int64_t k_ld,
                         const DropParams& dp, void* prob, void* alpha, hipStream_t st) {
    AttnArgs g{};
    g.a = attn_op(q, q_outer, q_inner, q_ld);
    g.b = attn_op(k, k_outer, k_inner, k_ld);
    g.B = B; g.H = H; g.J = J; g.K = K; g.D = D;
    g.out_scale = scaler; g.sm_scale = 1.0f; g.dp = dp;
    g.out0 = prob; g.out1 = alpha;
    if (dtype == DM_F16) attn_fused_t<half_t, false>(g, st);
    else attn_fused_t<bf16_t, false>(g, st);
}

void run_attn_scores_bwd(int dtype, int B, int H, int J, int K, int D, float scaler, const void* dgamma,
                         int64_t dg_outer, int64_t dg_inner, int64_t dg_ld, const void* v, int64_t v_outer,
                         int64_t v_inner, int64_t v_ld, const void* prob, const DropParams& dp, void* dbeta,
                         hipStream_t st) {
    AttnArgs g{};
    g.a = attn_op(dgamma, dg_outer, dg_inner, dg_ld);
    g.b = attn_op(v, v_outer, v_inner, v_ld);
    g.B = B; g.H = H; g.J = J; g.K = K; g.D = D;
    g.out_scale = 1.0f; g.sm_scale = scaler; g.dp = dp;
    g.prob = prob; g.out0 = dbeta;
    if (dtype == DM_F16) attn_fused_t<half_t, true>(g, st);
    else attn_fused_t<bf16_t, true>(g, st);
}

}  // namespace dm
