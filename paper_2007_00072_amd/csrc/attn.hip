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
                    V8<T>::store(reinterpret_cast<T*>(g.out0) + base + col, v[i]);
                    dropout8(g.dp, (uint64_t)(ebase + col), v[i]);
                    const u32x4 pk = V8<T>::pack(v[i]);
                    *reinterpret_cast<u32x4*>(reinterpret_cast<T*>(g.out1) + base + col) = pk;
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
            T* obase = const_cast<T*>(reinterpret_cast<const T*>(g.o2.ptr)) + b * g.o2.outer + h * g.o2.inner + cbn * 32 + c;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int j = j0 + 8 * (r >> 2) + 4 * hh + (r & 3);
                if (j < J) obase[(int64_t)j * g.o2.ld] = from_f<T>(acc[r]);
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
