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
// Optionally the same block then runs the next contraction of the 32 rows
// it holds, reading the just-rounded row tile from LDS instead of HBM:
// forward gamma = alpha V (Table 3 row Gamma), backward
// dQ = d(beta) K (row QK^T dX1).  The key-side operand [k][n] (V or K) is
// n-contiguous, so each wave stages 16 x 32 pieces of it in a private LDS
// slot and reads them k-contiguous with the gfx950 transposing read.  The
// waves split the k steps, and the partial sums are added in a fixed order.
//
// The MFMA operands come straight from global memory: lane l of a 32x32x16
// step holds row l % 32 of its operand at 8 contraction indices, and since
// the sum over the contraction index may run in any order, the lanes of
// half-wave hh take indices [hh D/2, (hh + 1) D/2) in D/16 steps of 8, i.e.
// each lane reads D/2 contiguous elements of its row.
#include <math.h>

#include <algorithm>

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

template <typename T>
__device__ __forceinline__ uint32_t bits16(T v) {
    return (uint32_t)__builtin_bit_cast(uint16_t, v);
}

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
    AttnOp x;            // second contraction: key-side rows [k][n] (V forward, K backward)
    AttnOp o2;           // its output: element (z, j, n) at ptr + b*outer + h*inner + j*ld + n
    float* o2f;          // optional fp32 copy of that output before rounding (same strides)
    int N2;              // its width (a multiple of 32), 0 when there is none
    int causal;          // forward: query j sees keys k <= j only
};

// One k16 step of the second contraction stages a 16 x 32 piece of the
// key-side operand: lane l holds row l / 4, elements 8 (l % 4) .. +7.
// Rows are 64 bytes, so the four rows that one transposing read touches in
// each half-wave cover the 64 banks once.
template <typename T>
__device__ __forceinline__ u32x4 stage_frag(const T* stg, int lane) {
    typedef short s4 __attribute__((ext_vector_type(4)));
    typedef __attribute__((address_space(3))) s4 lds_s4;
    // lanes 16g .. 16g+15 receive column 16 (g % 2) + l % 16 at k = 8 (g / 2) .. +7
    const int gq = lane >> 4, sl = lane & 15;
    const T* p = stg + (8 * (gq >> 1) + (sl >> 2)) * 32 + 16 * (gq & 1) + 4 * (sl & 3);
    const s4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4*)p);
    const s4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4*)(p + 4 * 32));
    u32x4 out;
    out[0] = (uint16_t)lo[0] | ((uint32_t)(uint16_t)lo[1] << 16);
    out[1] = (uint16_t)lo[2] | ((uint32_t)(uint16_t)lo[3] << 16);
    out[2] = (uint16_t)hi[0] | ((uint32_t)(uint16_t)hi[1] << 16);
    out[3] = (uint16_t)hi[2] | ((uint32_t)(uint16_t)hi[3] << 16);
    return out;
}

constexpr int STG_BYTES = 2048;  // per-wave staging slot: two 16 x 32 pieces
constexpr int PF2 = 8;           // k16 steps of the second contraction loaded ahead into registers

// chunk permutation mask of the score tile's rows (K a multiple of 8)
__host__ __device__ inline int tile_swizzle_mask(int K) {
    const int ch = K / 8, low = ch & -ch;
    return (low < 16 ? low : 16) - 1;
}

inline size_t attn_lds_bytes(int K, int es, int nb2) {
    const size_t s = (size_t)32 * K * es;
    if (nb2 == 0) return s;
    const size_t ks = 8 / nb2;
    return std::max(s + (size_t)(NTA / 64) * STG_BYTES, (ks - 1) * nb2 * 4096);
}

template <typename T, int LPR, int NV, int DK, bool BWD, int NB2>
__global__ __launch_bounds__(NTA) void attn_fused_k(AttnArgs g) {
    extern __shared__ __attribute__((aligned(16))) unsigned char smem_raw[];
    T* S = reinterpret_cast<T*>(smem_raw);
    // unpadded rows of K elements; the 16-byte chunks of row r are permuted
    // by chunk ^ (r & swm) (swm + 1 = the largest power of two up to 16
    // dividing K / 8), so the 8-byte tile writes, the 16-byte fragment reads
    // and the row operator's 16-byte accesses spread over the 64 banks as
    // padded rows would, while the tile takes no more than 32 K elements
    const int K = g.K, J = g.J, swm = tile_swizzle_mask(K);
    auto at = [&](int r, int col) { return r * K + ((((col >> 3) ^ (r & swm))) << 3) + (col & 7); };
    // Workgroups reach the 8 XCDs round-robin by linear id; the row blocks
    // of one (b, h) are given consecutive ids within one XCD's share, so
    // that XCD's L2 serves the head's key-side rows to all of them
    // instead of each XCD fetching every head's rows.
    const int nrb = (int)gridDim.x, nblocks = nrb * (int)gridDim.y;
    int lid = (int)blockIdx.y * nrb + (int)blockIdx.x;
    if ((nblocks & 7) == 0) lid = (lid & 7) * (nblocks >> 3) + (lid >> 3);
    const int z = lid / nrb, j0 = (lid - z * nrb) * 32;
    const int b = z / g.H, h = z - b * g.H;
    const int tid = threadIdx.x, lane = tid & 63, c = lane & 31, hh = lane >> 5;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);

    // row phase geometry: one lane group of LPR lanes per row, NV 8-element
    // vectors per lane, NIT rows per lane group
    constexpr int RPW = 64 / LPR;
    constexpr int NIT = (32 + (NTA / 64) * RPW - 1) / ((NTA / 64) * RPW);  // lane groups past row 31 stay idle
    const int gi = lane / LPR, gl = lane % LPR;
    const int nr = min(32, J - j0);

    // backward: the rows of P this lane reads start loading now and arrive
    // while the first contraction runs (clamped to valid rows and columns;
    // what lies outside is never used)
    [[maybe_unused]] u32x4 pre[BWD ? NIT : 1][NV];
    if constexpr (BWD) {
#pragma unroll
        for (int it = 0; it < NIT; ++it) {
            const int jj = min(j0 + it * (NTA / 64) * RPW + wave * RPW + gi, J - 1);
#pragma unroll
            for (int i = 0; i < NV; ++i)
                pre[it][i] = *reinterpret_cast<const u32x4*>(reinterpret_cast<const T*>(g.prob) +
                                                             ((int64_t)z * J + jj) * K + min((gl + i * LPR) * 8, K - 8));
        }
    }

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
            // key rows as the MFMA's first operand: the result is the tile's
            // transpose, so lane l holds query row l % 32 at 4 consecutive
            // keys per accumulator quad and writes them as one 8-byte piece
#pragma unroll
            for (int s = 0; s < DK; ++s) acc = AMfma<T>::run(bf[s], af[s], acc);
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                uint2 pk;
                pk.x = bits16(from_f<T>(acc[4 * q] * g.out_scale)) | (bits16(from_f<T>(acc[4 * q + 1] * g.out_scale)) << 16);
                pk.y = bits16(from_f<T>(acc[4 * q + 2] * g.out_scale)) |
                       (bits16(from_f<T>(acc[4 * q + 3] * g.out_scale)) << 16);
                *reinterpret_cast<uint2*>(S + at(c, cb * 32 + 8 * q + 4 * hh)) = pk;
            }
        }
    }
    __syncthreads();

    // ---- second contraction, part 1: its key-side rows start loading
    // before the row phase forward (arriving while it runs) and right after
    // it backward (where P's preloaded rows hold the registers until then).
    // Wave w takes output columns 32 (w % NB2) .. +31 and the k16 steps
    // s = w / NB2 + KS i.
    constexpr int KS = NB2 > 0 ? 8 / NB2 : 1;
    const int cbn = NB2 > 0 ? wave % NB2 : 0, ks = NB2 > 0 ? wave / NB2 : 0;
    const int nst = K / 16;
    const int cnt = (NB2 > 0 && ks < KS) ? (nst - ks + KS - 1) / KS : 0;
    [[maybe_unused]] u32x4 xr[NB2 > 0 ? PF2 : 1];
    [[maybe_unused]] const T* xbase = nullptr;
    // every wave loads (idle ones and steps past the end re-read the last step)
    auto load_next = [&](int g0) {
#pragma unroll
        for (int i = 0; i < PF2; ++i)
            xr[i] = *reinterpret_cast<const u32x4*>(xbase + (int64_t)(16 * min(ks + KS * (g0 + i), nst - 1) +
                                                                       (lane >> 2)) * g.x.ld);
    };
    if constexpr (NB2 > 0) {
        xbase = reinterpret_cast<const T*>(g.x.ptr) + b * g.x.outer + h * g.x.inner + cbn * 32 + 8 * (lane & 3);
        if constexpr (!BWD) load_next(0);
    }

    // ---- row phase
#pragma unroll
    for (int it = 0; it < NIT; ++it) {
        const int lr = it * (NTA / 64) * RPW + wave * RPW + gi;
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
                    V8<T>::unpack(*reinterpret_cast<const u32x4*>(S + at(lr, col)), v[i]);
                    if (g.causal) {
#pragma unroll
                        for (int q = 0; q < 8; ++q)
                            if (col + q > j) v[i][q] = -INFINITY;  // keys after the query (probability 0)
                    }
#pragma unroll
                    for (int q = 0; q < 8; ++q) mx = fmaxf(mx, v[i][q]);
                } else {
#pragma unroll
                    for (int q = 0; q < 8; ++q) v[i][q] = -INFINITY;
                }
            }
            mx = group_max<LPR>(mx);
            float sum = 0.f;
            const ExpShift ex(mx);
#pragma unroll
            for (int i = 0; i < NV; ++i)
#pragma unroll
                for (int q = 0; q < 8; ++q) { v[i][q] = ex(v[i][q]); sum += v[i][q]; }
            sum = group_sum<LPR>(sum);
            if (!active) continue;
            const float rinv = __builtin_amdgcn_rcpf(sum);
#pragma unroll
            for (int i = 0; i < NV; ++i) {
                const int col = (gl + i * LPR) * 8;
                if (col < K) {
#pragma unroll
                    for (int q = 0; q < 8; ++q) v[i][q] *= rinv;
                    // alpha is the dropout of P as stored (rounded)
                    const u32x4 pp = V8<T>::pack(v[i]);
                    *reinterpret_cast<u32x4*>(reinterpret_cast<T*>(g.out0) + base + col) = pp;
                    V8<T>::unpack(pp, v[i]);
                    dropout8(g.dp, (uint64_t)(ebase + col), v[i]);
                    const u32x4 pk = V8<T>::pack(v[i]);
                    if (g.out1) *reinterpret_cast<u32x4*>(reinterpret_cast<T*>(g.out1) + base + col) = pk;
                    if constexpr (NB2 > 0) *reinterpret_cast<u32x4*>(S + at(lr, col)) = pk;
                }
            }
        } else {
            float p[NV][8];
            float dot = 0.f;
#pragma unroll
            for (int i = 0; i < NV; ++i) {
                const int col = (gl + i * LPR) * 8;
                if (active && col < K) {
                    V8<T>::unpack(pre[it][i], p[i]);
                    V8<T>::unpack(*reinterpret_cast<const u32x4*>(S + at(lr, col)), v[i]);
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
                    const u32x4 pk = V8<T>::pack(o);
                    *reinterpret_cast<u32x4*>(reinterpret_cast<T*>(g.out0) + base + col) = pk;
                    if constexpr (NB2 > 0) *reinterpret_cast<u32x4*>(S + at(lr, col)) = pk;
                }
            }
        }
    }

    // ---- second contraction, part 2: out2[j][n] = sum_k S[j][k] X[k][n] over
    // the rounded row tile now in LDS (alpha forward, d(beta) backward)
    if constexpr (NB2 > 0) {
        if constexpr (BWD) load_next(0);
        __syncthreads();
        const size_t s_bytes = (size_t)32 * K * sizeof(T);
        T* stg = reinterpret_cast<T*>(smem_raw + s_bytes + wave * STG_BYTES);
        floatx16 acc;
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[r] = 0.f;

        for (int g0 = 0; g0 < cnt; g0 += PF2) {
            if (g0 > 0) load_next(g0);
#pragma unroll
            for (int i = 0; i < PF2; i += 2) {
                if (g0 + i < cnt) {
                    // the slot's previous reads were issued before these writes, and
                    // one wave's LDS operations complete in order
                    *reinterpret_cast<u32x4*>(stg + (lane >> 2) * 32 + 8 * (lane & 3)) = xr[i];
                    if (g0 + i + 1 < cnt)
                        *reinterpret_cast<u32x4*>(stg + 512 + (lane >> 2) * 32 + 8 * (lane & 3)) = xr[i + 1];
                    const int s0 = 16 * (ks + KS * (g0 + i));
                    acc = AMfma<T>::run(*reinterpret_cast<const u32x4*>(S + at(c, s0 + 8 * hh)), stage_frag(stg, lane), acc);
                    if (g0 + i + 1 < cnt) {
                        const int s1 = 16 * (ks + KS * (g0 + i + 1));
                        acc = AMfma<T>::run(*reinterpret_cast<const u32x4*>(S + at(c, s1 + 8 * hh)), stage_frag(stg + 512, lane),
                                            acc);
                    }
                }
            }
        }
        __syncthreads();  // every wave is done with the row tile and its slot
        float* red = reinterpret_cast<float*>(smem_raw);
        if (ks > 0 && ks < KS) {
#pragma unroll
            for (int r = 0; r < 16; ++r) red[((ks - 1) * NB2 + cbn) * 1024 + r * 64 + lane] = acc[r];
        }
        __syncthreads();
        if (ks == 0) {
#pragma unroll 1
            for (int q = 1; q < KS; ++q) {
#pragma unroll
                for (int r = 0; r < 16; ++r) acc[r] += red[((q - 1) * NB2 + cbn) * 1024 + r * 64 + lane];
            }
            const int64_t ooff = b * g.o2.outer + h * g.o2.inner + cbn * 32 + c;
            T* obase = const_cast<T*>(reinterpret_cast<const T*>(g.o2.ptr)) + ooff;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int j = j0 + 8 * (r >> 2) + 4 * hh + (r & 3);
                if (j < J) obase[(int64_t)j * g.o2.ld] = from_f<T>(acc[r]);
            }
            if (g.o2f) {
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int j = j0 + 8 * (r >> 2) + 4 * hh + (r & 3);
                    if (j < J) g.o2f[ooff + (int64_t)j * g.o2.ld] = acc[r];
                }
            }
        }
    }
}

template <typename T, bool BWD, int LPR, int NV, int DK>
void attn_fused_d(const AttnArgs& g, hipStream_t st) {
    const dim3 grid((g.J + 31) / 32, g.B * g.H);
    const int nb2 = g.N2 / 32;
    const size_t lds = attn_lds_bytes(g.K, (int)sizeof(T), nb2);
    if constexpr (DK == 2 || DK == 4 || DK == 8) {
        switch (nb2) {
            case 1: hipLaunchKernelGGL((attn_fused_k<T, LPR, NV, DK, BWD, 1>), grid, dim3(NTA), lds, st, g); return;
            case 2: hipLaunchKernelGGL((attn_fused_k<T, LPR, NV, DK, BWD, 2>), grid, dim3(NTA), lds, st, g); return;
            case 4: hipLaunchKernelGGL((attn_fused_k<T, LPR, NV, DK, BWD, 4>), grid, dim3(NTA), lds, st, g); return;
            default: break;
        }
    }
    hipLaunchKernelGGL((attn_fused_k<T, LPR, NV, DK, BWD, 0>), grid, dim3(NTA), lds, st, g);
}

// N2 is 0 here unless attn_next_ok admitted it (D and N2 in {32, 64, 128})
template <typename T, bool BWD, int LPR, int NV>
void attn_fused_n(const AttnArgs& g, hipStream_t st) {
    switch (g.D / 16) {
        case 1: attn_fused_d<T, BWD, LPR, NV, 1>(g, st); break;
        case 2: attn_fused_d<T, BWD, LPR, NV, 2>(g, st); break;
        case 3: attn_fused_d<T, BWD, LPR, NV, 3>(g, st); break;
        case 4: attn_fused_d<T, BWD, LPR, NV, 4>(g, st); break;
        case 6: attn_fused_d<T, BWD, LPR, NV, 6>(g, st); break;
        default: attn_fused_d<T, BWD, LPR, NV, 8>(g, st); break;
    }
}

template <typename T, bool BWD>
void attn_fused_t(const AttnArgs& g, hipStream_t st) {
    const int len = g.K;
    if (len <= 32) attn_fused_n<T, BWD, 4, 1>(g, st);
    else if (len <= 64) attn_fused_n<T, BWD, 8, 1>(g, st);
    else if (len <= 128) attn_fused_n<T, BWD, 16, 1>(g, st);
    else if (len <= 256) attn_fused_n<T, BWD, 32, 1>(g, st);
    else if (len <= 512) attn_fused_n<T, BWD, 64, 1>(g, st);
    else attn_fused_n<T, BWD, 64, 2>(g, st);
}

// ---------------------------------------------------------------------------
// Key-block backward: Table 3 rows Gamma dX1 (d(alpha)), `bs`, Gamma dX2
// (dV), QK^T dX1 (dQ) and QK^T dX2 (dK) in one launch that reads the
// scores' only saved tensor, P, once and writes none of d(alpha), alpha or
// d(beta).  A block owns KB = 32 KG keys of one (b, h) and walks the query
// rows JB = 32 QG at a time (KG QG = 8 waves; wave (qg, kg) takes query
// rows 32 qg.. and keys 32 kg.. of each step):
//   d(alpha)^T tile on MFMA from this wave's V rows (held in registers) and
//     the step's d(gamma) rows (staged in LDS); each lane then holds 16
//     consecutive keys of one query row;
//   the row operator regenerates the dropout keep decisions of those 16
//     keys (4 Philox draws), forms alpha = dropout(P) exactly as the forward
//     did from the stored P, and d(beta) = s P (dP - D_j) with
//     dP = dropout(d(alpha)) (d(alpha) in fp32, never stored) and the row
//     term D_j = sum_k d(alpha)_jk alpha_jk (= sum_k dP P), which equals
//     d(gamma)_j . gamma_j with gamma = alpha V before rounding (saved in
//     fp32 by the forward) and needs the row's 64 head values instead of
//     all K scores;
//   alpha and d(beta) go to LDS; dV += alpha^T d(gamma) and
//     dK += d(beta)^T Q accumulate over all query steps in registers, their
//     operands read k-contiguous with the gfx950 transposing LDS read;
//   dQ = d(beta) K for the step's rows: each wave takes one 32 x 32 output
//     tile over a 64-key chunk (K fragments held in registers); the chunks'
//     fp32 tiles meet in LDS, where every wave adds up (in chunk order) and
//     stores an equal share of the step's rows.
// With more than one key block per head (nkb > 1) the block's dQ rows are
// an fp32 partial over its keys, added in key-block order by
// attn_dq_reduce_k; the sums are deterministic either way.
constexpr int KV_HD = 64;  // head size (P = W) of the key-block backward

struct KeysArgs {
    AttnOp q, k, v;   // rows [z][row][64]
    AttnOp dg, gm;    // d(gamma), fp32 gamma: token rows (z, j) -> b*outer + h*inner + j*ld
    const void* prob; // P [B][H][J][K]
    DropParams dp;
    float sm_scale;
    int B, H, J, K, nkb;
    AttnOp dq, dk, dv;  // outputs (dq written only when nkb == 1)
    float* part;        // nkb > 1: dQ partials [nkb][B*H][J][64]
};

typedef short s4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s4_t lds_s4_t;

__device__ __forceinline__ u32x4 join_tr(s4_t lo, s4_t hi) {
    u32x4 out;
    out[0] = (uint16_t)lo[0] | ((uint32_t)(uint16_t)lo[1] << 16);
    out[1] = (uint16_t)lo[2] | ((uint32_t)(uint16_t)lo[3] << 16);
    out[2] = (uint16_t)hi[0] | ((uint32_t)(uint16_t)hi[1] << 16);
    out[3] = (uint16_t)hi[2] | ((uint32_t)(uint16_t)hi[3] << 16);
    return out;
}

// LDS tiles of 16-bit elements, addressed in bytes.  Rows of the [JB][KB]
// alpha / d(beta) tiles permute their 16-byte chunks by
// chunk ^ (4 (r & 3) + ((r >> 2) & 3)): the row operator's 16-byte writes
// (32 rows at one chunk) and the transposing reads (4 + 4 rows at 4
// chunks) both reach every bank evenly.  Rows of 64 elements (the staged
// d(gamma), Q and K tiles) permute by chunk ^ ((r >> 1) & 7).
template <int ROWB>
__device__ __forceinline__ int ab_off(int r, int col) {
    return r * ROWB + ((((col >> 3) ^ (4 * (r & 3) + ((r >> 2) & 3)))) << 4) + ((col & 7) << 1);
}
__device__ __forceinline__ int hd_off(int r, int col) {
    return r * 128 + ((((col >> 3) ^ ((r >> 1) & 7))) << 4) + ((col & 7) << 1);
}

template <typename T, int KG>
__global__ __launch_bounds__(NTA) void attn_bwd_keys_k(KeysArgs g) {
    constexpr int QG = 8 / KG, KB = 32 * KG, JB = 32 * QG;
    constexpr int NT2 = 2 * QG;   // dQ tiles (32 x 32) per step
    constexpr int NCH = 8 / NT2;  // 64-key chunks per dQ tile
    static_assert(NCH * 64 == KB, "dQ chunks");
    constexpr int ROWB = KB * 2;
    constexpr int AB = JB * ROWB;  // bytes of the alpha tile (as of d(beta))
    constexpr int HDT = JB * 128;  // bytes of one staged [JB][64] tile
    // two staging buffers (one step's d(gamma) and Q rows and D values):
    // the row operator of step i writes step i + 1's while step i's are read
    constexpr int SB = 2 * HDT + JB * 4;
    constexpr int OFF_A = 0, OFF_DB = AB, OFF_STG = 2 * AB;
    constexpr int OFF_RED = OFF_STG + 2 * SB;
    constexpr int LDS = OFF_RED + NCH * NT2 * 4096;
    // the K staging and the final query-group sums reuse the alpha / d(beta) tiles
    static_assert(KB * 128 <= 2 * AB && (QG - 1) * KG * 2 * 4096 <= 2 * AB, "LDS reuse");
    __shared__ __attribute__((aligned(16))) unsigned char lds[LDS];

    const int nz = g.B * g.H;
    const int nblk = (int)gridDim.x * (int)gridDim.y;
    int lid = (int)blockIdx.y * (int)gridDim.x + (int)blockIdx.x;
    // the key blocks of one head run on one XCD (see attn_fused_k)
    if ((nblk & 7) == 0) lid = (lid & 7) * (nblk >> 3) + (lid >> 3);
    const int z = lid / g.nkb, kb = lid - z * g.nkb;
    const int b = z / g.H, h = z - b * g.H;
    const int k0 = kb * KB;
    const int tid = threadIdx.x, lane = tid & 63, c32 = lane & 31, hh = lane >> 5;
    const int grp = lane >> 4, sl = lane & 15;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int qg = wave / KG, kg = wave - qg * KG;
    const int tq = wave % NT2, qt = tq >> 1, pt = tq & 1, ch = wave / NT2;  // dQ task

    const T* Qz = reinterpret_cast<const T*>(g.q.ptr) + b * g.q.outer + h * g.q.inner;
    const T* Kz = reinterpret_cast<const T*>(g.k.ptr) + b * g.k.outer + h * g.k.inner;
    const T* Vz = reinterpret_cast<const T*>(g.v.ptr) + b * g.v.outer + h * g.v.inner;
    const T* DGz = reinterpret_cast<const T*>(g.dg.ptr) + b * g.dg.outer + h * g.dg.inner;
    const float* GMz = reinterpret_cast<const float*>(g.gm.ptr) + b * g.gm.outer + h * g.gm.inner;
    const T* Pz = reinterpret_cast<const T*>(g.prob) + (int64_t)z * g.J * g.K;

    auto tr = [&](int off) { return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4_t*)(lds + off)); };
    // k-contiguous fragment of rows rs + 8 hh .. +7 at column ctile + lane % 32
    auto frag_ab = [&](int base, int rs, int ctile) {
        const int r = rs + 8 * hh + (sl >> 2), c = ctile + 16 * (grp & 1) + 4 * (sl & 3);
        return join_tr(tr(base + ab_off<ROWB>(r, c)), tr(base + ab_off<ROWB>(r + 4, c)));
    };
    auto frag_hd = [&](int base, int rs, int ctile) {
        const int r = rs + 8 * hh + (sl >> 2), c = ctile + 16 * (grp & 1) + 4 * (sl & 3);
        return join_tr(tr(base + hd_off(r, c)), tr(base + hd_off(r + 4, c)));
    };

    // V rows of this wave's keys, the first operand of d(alpha)^T: MFMA row
    // m = 8 q + 4 e + i takes key 16 e + 4 q + i, so that the result gives
    // lane half hh the 16 consecutive keys 16 hh .. +15
    u32x4 vf[4];
    {
        const int key = k0 + 32 * kg + 16 * ((c32 >> 2) & 1) + 4 * (c32 >> 3) + (c32 & 3);
        const T* vr = Vz + (int64_t)key * g.v.ld + 32 * hh;
#pragma unroll
        for (int s = 0; s < 4; ++s) vf[s] = *reinterpret_cast<const u32x4*>(vr + 8 * s);
    }
    // K rows of the block, staged once for the dQ fragments
    for (int pc = tid; pc < KB * 8; pc += NTA) {
        const int r = pc >> 3, c = (pc & 7) * 8;
        *reinterpret_cast<u32x4*>(lds + OFF_A + hd_off(r, c)) =
            *reinterpret_cast<const u32x4*>(Kz + (int64_t)(k0 + r) * g.k.ld + c);
    }

    // staging of one step's d(gamma) and Q rows (and D = d(gamma) . gamma):
    // thread t < JB * 8 moves 16 bytes of row t / 8
    const bool stager = tid < JB * 8;
    const int srow = tid >> 3, sc = (tid & 7) * 8;
    u32x4 sdg = {0, 0, 0, 0}, sq = {0, 0, 0, 0};
    floatx4 sgm0 = {0.f, 0.f, 0.f, 0.f}, sgm1 = {0.f, 0.f, 0.f, 0.f};
    auto stage_load = [&](int j0) {
        if (!stager) return;
        const int j = min(j0 + srow, g.J - 1);
        sdg = *reinterpret_cast<const u32x4*>(DGz + (int64_t)j * g.dg.ld + sc);
        sgm0 = *reinterpret_cast<const floatx4*>(GMz + (int64_t)j * g.gm.ld + sc);
        sgm1 = *reinterpret_cast<const floatx4*>(GMz + (int64_t)j * g.gm.ld + sc + 4);
        sq = *reinterpret_cast<const u32x4*>(Qz + (int64_t)j * g.q.ld + sc);
    };
    auto stage_store = [&](int j0, int buf) {
        const int OFF_DG = OFF_STG + buf * SB, OFF_Q = OFF_DG + HDT, OFF_D = OFF_Q + HDT;
        float dd = 0.f;
        if (stager) {
            if (j0 + srow >= g.J) {  // rows past the end are zeros
                sdg = u32x4{0, 0, 0, 0};
                sq = u32x4{0, 0, 0, 0};
            }
            float a[8];
            V8<T>::unpack(sdg, a);
#pragma unroll
            for (int i = 0; i < 4; ++i) dd = fmaf(a[i], sgm0[i], dd);
#pragma unroll
            for (int i = 0; i < 4; ++i) dd = fmaf(a[4 + i], sgm1[i], dd);
            *reinterpret_cast<u32x4*>(lds + OFF_DG + hd_off(srow, sc)) = sdg;
            *reinterpret_cast<u32x4*>(lds + OFF_Q + hd_off(srow, sc)) = sq;
        }
        dd = group_sum<8>(dd);
        if (stager && sc == 0) *reinterpret_cast<float*>(lds + OFF_D + 4 * srow) = dd;
    };
    // P of this lane's 16 keys in query row j0 + 32 qg + lane % 32
    u32x4 pf[2];
    auto p_load = [&](int j0) {
        const int j = min(j0 + 32 * qg + c32, g.J - 1);
        const T* pr = Pz + (int64_t)j * g.K + k0 + 32 * kg + 16 * hh;
        pf[0] = *reinterpret_cast<const u32x4*>(pr);
        pf[1] = *reinterpret_cast<const u32x4*>(pr + 8);
    };
    const int nit = (g.J + JB - 1) / JB;
    stage_load(0);
    p_load(0);
    __syncthreads();
    // dQ task: rows of tile qt, columns 32 pt .., keys 64 ch + 16 s + 8 hh + t
    u32x4 kf[4];
#pragma unroll
    for (int s = 0; s < 4; ++s) kf[s] = frag_hd(OFF_A, 64 * ch + 16 * s, 32 * pt);
    stage_store(0, 0);
    if (nit > 1) stage_load(JB);
    __syncthreads();

    floatx16 accV[2], accK[2];
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) { accV[t][r] = 0.f; accK[t][r] = 0.f; }
    const int64_t erow0 = ((int64_t)h * g.B + b) * g.J;  // dropout logical row of (h, b, j = 0)
    const bool drop = g.dp.enabled != 0;
    const float dscale = drop ? g.dp.scale : 1.0f;
    const uint32_t thr = (uint32_t)g.dp.thr;
    const uint32_t sk0 = (uint32_t)g.dp.seed, sk1 = (uint32_t)(g.dp.seed >> 32);
    float* red = reinterpret_cast<float*>(lds + OFF_RED);
    const int kl = 32 * kg + 16 * hh;  // first key (within the block) of this lane's row piece

    for (int it = 0; it < nit; ++it) {
        const int j0 = it * JB;
        const int OFF_DG = OFF_STG + (it & 1) * SB, OFF_Q = OFF_DG + HDT, OFF_D = OFF_Q + HDT;
        // ---- d(alpha)^T: 32 keys x 32 queries
        floatx16 da;
#pragma unroll
        for (int r = 0; r < 16; ++r) da[r] = 0.f;
#pragma unroll
        for (int s = 0; s < 4; ++s)
            da = AMfma<T>::run(vf[s], *reinterpret_cast<const u32x4*>(lds + OFF_DG + hd_off(32 * qg + c32, 32 * hh + 8 * s)),
                               da);
        // ---- row operator: da[r] = d(alpha) of query row j at key k0 + kl + r
        const int jl = 32 * qg + c32, j = j0 + jl;
        const bool valid = j < g.J;
        float p[16];
        V8<T>::unpack(pf[0], p);
        V8<T>::unpack(pf[1], p + 8);
        const float Dj = *reinterpret_cast<const float*>(lds + OFF_D + 4 * jl);
        const uint64_t blk0 = ((uint64_t)(erow0 + j) * (uint64_t)g.K + (uint64_t)(k0 + kl)) >> 2;
        float al[16], db[16];
        // the four draws in one straight run, so their round chains interleave
        u32x4 w[4];
        if (drop) {
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const uint64_t blk = blk0 + q;
                w[q] = Philox::gen((uint32_t)blk, (uint32_t)(blk >> 32), g.dp.site, g.dp.layer, sk0, sk1);
            }
        } else {
#pragma unroll
            for (int q = 0; q < 4; ++q) w[q] = u32x4{0, 0, 0, 0};
        }
#pragma unroll
        for (int q = 0; q < 4; ++q) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int r = 4 * q + i;
                const float pv = valid ? p[r] : 0.f;
                const bool keep = !drop || w[q][i] < thr;
                const float dpv = keep ? da[r] * dscale : 0.f;
                db[r] = g.sm_scale * pv * (dpv - Dj);
                al[r] = keep ? pv * dscale : 0.f;
            }
        }
        *reinterpret_cast<u32x4*>(lds + OFF_A + ab_off<ROWB>(jl, kl)) = V8<T>::pack(al);
        *reinterpret_cast<u32x4*>(lds + OFF_A + ab_off<ROWB>(jl, kl + 8)) = V8<T>::pack(al + 8);
        *reinterpret_cast<u32x4*>(lds + OFF_DB + ab_off<ROWB>(jl, kl)) = V8<T>::pack(db);
        *reinterpret_cast<u32x4*>(lds + OFF_DB + ab_off<ROWB>(jl, kl + 8)) = V8<T>::pack(db + 8);
        // next step: its staged rows (loaded one step ahead) into the other
        // buffer, then the loads for the step after
        if (it + 1 < nit) {
            stage_store(j0 + JB, (it + 1) & 1);
            p_load(j0 + JB);
            if (it + 2 < nit) stage_load(j0 + 2 * JB);
        }
        __syncthreads();

        // ---- dV += alpha^T d(gamma), dK += d(beta)^T Q over this wave's 32 queries
#pragma unroll
        for (int s = 0; s < 2; ++s) {
            const int rs = 32 * qg + 16 * s;
            const u32x4 fa = frag_ab(OFF_A, rs, 32 * kg), fb = frag_ab(OFF_DB, rs, 32 * kg);
#pragma unroll
            for (int t = 0; t < 2; ++t) {
                accV[t] = AMfma<T>::run(fa, frag_hd(OFF_DG, rs, 32 * t), accV[t]);
                accK[t] = AMfma<T>::run(fb, frag_hd(OFF_Q, rs, 32 * t), accK[t]);
            }
        }
        // ---- dQ tile (qt, pt) over keys 64 ch .. +63
        floatx16 aq;
#pragma unroll
        for (int r = 0; r < 16; ++r) aq[r] = 0.f;
#pragma unroll
        for (int s = 0; s < 4; ++s)
            aq = AMfma<T>::run(*reinterpret_cast<const u32x4*>(lds + OFF_DB + ab_off<ROWB>(32 * qt + c32, 64 * ch + 16 * s + 8 * hh)),
                               kf[s], aq);
#pragma unroll
        for (int r = 0; r < 16; ++r) red[(ch * NT2 + tq) * 1024 + r * 64 + lane] = aq[r];
        __syncthreads();
        // every wave adds up (in chunk order) and stores 16 / NCH accumulator
        // rows of one dQ tile: wave w takes tile w % NT2, rows part w / NT2
        {
            constexpr int RPP = 16 / NCH;
            const int tt = wave % NT2, part = wave / NT2;
            const int pc = 32 * (tt & 1) + c32;
            float v[RPP];
#pragma unroll
            for (int i = 0; i < RPP; ++i) {
                const int r = part * RPP + i;
                v[i] = red[tt * 1024 + r * 64 + lane];
#pragma unroll
                for (int c2 = 1; c2 < NCH; ++c2) v[i] += red[(c2 * NT2 + tt) * 1024 + r * 64 + lane];
            }
            const int jrow = j0 + 32 * (tt >> 1) + 4 * hh;  // row of accumulator r: + 8 (r / 4) + r % 4
            const bool full = j0 + JB <= g.J;
            if (g.nkb == 1) {
                T* dst = reinterpret_cast<T*>(const_cast<void*>(g.dq.ptr)) + b * g.dq.outer + h * g.dq.inner + pc;
#pragma unroll
                for (int i = 0; i < RPP; ++i) {
                    const int r = part * RPP + i, jq = jrow + 8 * (r >> 2) + (r & 3);
                    if (full || jq < g.J) dst[(int64_t)jq * g.dq.ld] = from_f<T>(v[i]);
                }
            } else {
                float* dst = g.part + ((int64_t)kb * nz + z) * g.J * KV_HD + pc;
#pragma unroll
                for (int i = 0; i < RPP; ++i) {
                    const int r = part * RPP + i, jq = jrow + 8 * (r >> 2) + (r & 3);
                    if (full || jq < g.J) dst[(int64_t)jq * KV_HD] = v[i];
                }
            }
        }
    }

    // ---- dV, dK of the block's keys (query groups added in order first)
    if constexpr (QG > 1) {
        float* r2 = reinterpret_cast<float*>(lds);
#pragma unroll
        for (int pass = 0; pass < 2; ++pass) {
            floatx16* acc = pass ? accK : accV;
            if (qg > 0) {
#pragma unroll
                for (int t = 0; t < 2; ++t)
#pragma unroll
                    for (int r = 0; r < 16; ++r) r2[(((qg - 1) * KG + kg) * 2 + t) * 1024 + r * 64 + lane] = acc[t][r];
            }
            __syncthreads();
            if (qg == 0) {
#pragma unroll 1
                for (int q2 = 1; q2 < QG; ++q2)
#pragma unroll
                    for (int t = 0; t < 2; ++t)
#pragma unroll
                        for (int r = 0; r < 16; ++r) acc[t][r] += r2[(((q2 - 1) * KG + kg) * 2 + t) * 1024 + r * 64 + lane];
            }
            __syncthreads();
        }
    }
    if (qg == 0) {
        T* dvz = reinterpret_cast<T*>(const_cast<void*>(g.dv.ptr)) + b * g.dv.outer + h * g.dv.inner;
        T* dkz = reinterpret_cast<T*>(const_cast<void*>(g.dk.ptr)) + b * g.dk.outer + h * g.dk.inner;
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int key = k0 + 32 * kg + 8 * (r >> 2) + 4 * hh + (r & 3);
                dvz[(int64_t)key * g.dv.ld + 32 * t + c32] = from_f<T>(accV[t][r]);
                dkz[(int64_t)key * g.dk.ld + 32 * t + c32] = from_f<T>(accK[t][r]);
            }
    }
}

// dQ = sum over the key blocks of their fp32 partials (in block order),
// rounded once; thread t handles 8 consecutive head values of one row.
template <typename T>
__global__ __launch_bounds__(256) void attn_dq_reduce_k(const float* __restrict__ part, int nkb, int B, int H,
                                                         int J, AttnOp dq) {
    const int64_t n = (int64_t)B * H * J * (KV_HD / 8);
    const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (t >= n) return;
    const int64_t row = t / (KV_HD / 8);  // (z, j)
    const int c = (int)(t % (KV_HD / 8)) * 8;
    const int z = (int)(row / J), j = (int)(row % J);
    const int b = z / H, h = z % H;
    const int64_t stride = (int64_t)B * H * J * KV_HD;
    const float* src = part + row * KV_HD + c;
    float v[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = 0.f;
    for (int k = 0; k < nkb; ++k) {
        const floatx4 a = *reinterpret_cast<const floatx4*>(src + k * stride);
        const floatx4 bb = *reinterpret_cast<const floatx4*>(src + k * stride + 4);
#pragma unroll
        for (int i = 0; i < 4; ++i) { v[i] += a[i]; v[4 + i] += bb[i]; }
    }
    T* out = reinterpret_cast<T*>(const_cast<void*>(dq.ptr)) + b * dq.outer + h * dq.inner + (int64_t)j * dq.ld + c;
    V8<T>::store(out, v);
}

AttnOp attn_op(const void* p, int64_t outer, int64_t inner, int64_t ld) {
    AttnOp o;
    o.ptr = p; o.outer = outer; o.inner = inner; o.ld = ld;
    return o;
}

}  // namespace

bool attn_fused_ok(int dtype, int K, int D) {
    // the score tile (32 rows of K elements) stays within 64 KB of LDS
    return (dtype == DM_F16 || dtype == DM_BF16) && K % 32 == 0 && K <= 960 &&
           (D == 16 || D == 32 || D == 48 || D == 64 || D == 96 || D == 128);
}

namespace {
// key tiles per block: 8 (256 keys) when K allows it and the grid still
// has about one block per CU, else 4 (128 keys)
int keys_kg(int B, int H, int K) {
    return (K % 256 == 0 && (int64_t)B * H * (K / 256) >= 192) ? 8 : 4;
}
AttnOp op_of(const AttnRows& r) { return attn_op(r.ptr, r.outer, r.inner, r.ld); }
}  // namespace

bool attn_keys_ok(int dtype, int K, int P, int W) {
    return (dtype == DM_F16 || dtype == DM_BF16) && P == KV_HD && W == KV_HD && K % 128 == 0;
}

size_t attn_keys_part_bytes(int B, int H, int J, int K) {
    const int nkb = K / (32 * keys_kg(B, H, K));
    return nkb > 1 ? (size_t)nkb * B * H * J * KV_HD * sizeof(float) : 0;
}

void run_attn_bwd_keys(int dtype, int B, int H, int J, int K, float scaler, AttnRows q, AttnRows k, AttnRows v,
                       AttnRows dgamma, AttnRows gamma, const void* prob, const DropParams& dp, AttnRows dq,
                       AttnRows dk, AttnRows dv, float* part, hipStream_t st) {
    const int kg = keys_kg(B, H, K), nkb = K / (32 * kg);
    KeysArgs g{};
    g.q = op_of(q); g.k = op_of(k); g.v = op_of(v); g.dg = op_of(dgamma); g.gm = op_of(gamma);
    g.prob = prob; g.dp = dp; g.sm_scale = scaler;
    g.B = B; g.H = H; g.J = J; g.K = K; g.nkb = nkb;
    g.dq = op_of(dq); g.dk = op_of(dk); g.dv = op_of(dv); g.part = part;
    const dim3 grid(nkb, B * H);
    if (dtype == DM_F16) {
        if (kg == 8) hipLaunchKernelGGL((attn_bwd_keys_k<half_t, 8>), grid, dim3(NTA), 0, st, g);
        else hipLaunchKernelGGL((attn_bwd_keys_k<half_t, 4>), grid, dim3(NTA), 0, st, g);
    } else {
        if (kg == 8) hipLaunchKernelGGL((attn_bwd_keys_k<bf16_t, 8>), grid, dim3(NTA), 0, st, g);
        else hipLaunchKernelGGL((attn_bwd_keys_k<bf16_t, 4>), grid, dim3(NTA), 0, st, g);
    }
    if (nkb > 1) {
        trace_next("dq_reduce");
        const int64_t n = (int64_t)B * H * J * (KV_HD / 8);
        const dim3 rg((unsigned)((n + 255) / 256));
        if (dtype == DM_F16) hipLaunchKernelGGL((attn_dq_reduce_k<half_t>), rg, dim3(256), 0, st, part, nkb, B, H, J, g.dq);
        else hipLaunchKernelGGL((attn_dq_reduce_k<bf16_t>), rg, dim3(256), 0, st, part, nkb, B, H, J, g.dq);
    }
}

bool attn_next_ok(int dtype, int K, int D, const AttnNext& n) {
    const int es = 2;
    return attn_fused_ok(dtype, K, D) && (D == 32 || D == 64 || D == 128) &&
           (n.N == 32 || n.N == 64 || n.N == 128) && n.x && n.out &&
           reinterpret_cast<uintptr_t>(n.x) % 16 == 0 && n.x_outer % 8 == 0 && n.x_inner % 8 == 0 &&
           n.x_ld % 8 == 0 && n.x_ld >= n.N && attn_lds_bytes(K, es, n.N / 32) <= 65536;
}

namespace {
void set_next(AttnArgs& g, const AttnNext* n) {
    if (!n) return;
    g.x = attn_op(n->x, n->x_outer, n->x_inner, n->x_ld);
    g.o2 = attn_op(n->out, n->o_outer, n->o_inner, n->o_ld);
    g.o2f = n->out_f32;
    g.N2 = n->N;
}
}  // namespace

void run_attn_scores_fwd(int dtype, int B, int H, int J, int K, int D, float scaler, const void* q, int64_t q_outer,
                         int64_t q_inner, int64_t q_ld, const void* k, int64_t k_outer, int64_t k_inner, int64_t k_ld,
                         const DropParams& dp, void* prob, void* alpha, const AttnNext* next, hipStream_t st,
                         int causal) {
    AttnArgs g{};
    set_next(g, next);
    g.causal = causal;
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
                         const AttnNext* next, hipStream_t st) {
    AttnArgs g{};
    set_next(g, next);
    g.a = attn_op(dgamma, dg_outer, dg_inner, dg_ld);
    g.b = attn_op(v, v_outer, v_inner, v_ld);
    g.B = B; g.H = H; g.J = J; g.K = K; g.D = D;
    g.out_scale = 1.0f; g.sm_scale = scaler; g.dp = dp;
    g.prob = prob; g.out0 = dbeta;
    if (dtype == DM_F16) attn_fused_t<half_t, true>(g, st);
    else attn_fused_t<bf16_t, true>(g, st);
}

}  // namespace dm
