// MFMA contraction kernel for gfx950 (fp16 / bf16 storage, fp32
// accumulation) and a plain fp32 kernel for float32 layers.
//
// Block tile BM x BN, k-step BK, 256 threads = 4 wave64s in a 2 x 2 grid of
// wave tiles.  Both operands are staged in LDS as [outer][k] (k contiguous,
// row padded by 8 elements so the 16-byte fragment reads of 16 consecutive
// rows hit distinct banks).  A k-contiguous operand is copied with 16-byte
// loads; an outer-contiguous operand is loaded 4 k-rows x 8 outer elements
// per thread and transposed in registers on its way to LDS, so every einsum
// layout reaches the same inner loop without a separate transpose pass.
// The next k-step's global loads are issued before the current step's
// MFMAs (register prefetch + LDS double buffer, one barrier per step).
// The epilogue stages the fp32 tile through LDS and writes 16-byte vectors
// along whichever output index is contiguous.
#include "gemm.hpp"
#include "internal.hpp"

namespace dm {

IdxMap make_map(uint32_t r0, uint32_t r1, int64_t s0, int64_t s1, int64_t s2) {
    IdxMap m{};
    m.r0 = r0; m.r1 = r1; m.s0 = s0; m.s1 = s1; m.s2 = s2;
    auto magic = [](uint32_t d, uint32_t& mul, uint32_t& shr) {
        if (d == 0) { mul = 0; shr = 0; return; }
        uint32_t l = 0;
        while ((1ull << l) < d) ++l;
        mul = (uint32_t)(((1ull << 32) * ((1ull << l) - d)) / d + 1);
        shr = l;
    };
    magic(r0, m.mul0, m.shr0);
    magic(r1, m.mul1, m.shr1);
    return m;
}

namespace {

constexpr int NT = 256;
constexpr int PAD = 8;

template <typename T> struct Mfma;
template <> struct Mfma<half_t> {
    typedef half8 frag;
    __device__ __forceinline__ static floatx4 run(frag a, frag b, floatx4 c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
    }
};
template <> struct Mfma<bf16_t> {
    typedef bf16x8 frag;
    __device__ __forceinline__ static floatx4 run(frag a, frag b, floatx4 c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
    }
};

// Loads one operand tile (R outer x BK) of k-step k0 into registers.
template <typename T, int R, int BK, bool KC>
struct TileLoader;

// k-contiguous: each thread owns NV 16-byte vectors; row pointers are fixed
// for the whole k loop.
template <typename T, int R, int BK>
struct TileLoader<T, R, BK, true> {
    static constexpr int VPR = BK / 8;
    static constexpr int NV = R * VPR / NT;
    static_assert(NV * NT == R * VPR, "tile / thread mismatch");
    const T* rowp[NV];
    u32x4 reg[NV];
    int kv;

    __device__ __forceinline__ void init(const Operand& op, int outer0, int outer_max, int64_t boff) {
        int tid = threadIdx.x;
        kv = tid % VPR;
#pragma unroll
        for (int i = 0; i < NV; ++i) {
            int r = tid / VPR + i * (NT / VPR);
            int o = outer0 + r;
            rowp[i] = nullptr;
            if (o < outer_max) {
                int seg = 0;
                int64_t off = map_off(op.row, (uint32_t)o, op.nseg, &seg);
                rowp[i] = reinterpret_cast<const T*>(op.ptr[seg]) + boff + off;
            }
        }
    }
    __device__ __forceinline__ void load(const Operand&, int k0, int K) {
        int k = k0 + kv * 8;
#pragma unroll
        for (int i = 0; i < NV; ++i) {
            u32x4 z = {0u, 0u, 0u, 0u};
            reg[i] = (rowp[i] && k < K) ? *reinterpret_cast<const u32x4*>(rowp[i] + k) : z;
        }
    }
    __device__ __forceinline__ void store(T* lds) {
        int tid = threadIdx.x;
#pragma unroll
        for (int i = 0; i < NV; ++i) {
            int r = tid / VPR + i * (NT / VPR);
            *reinterpret_cast<u32x4*>(lds + r * (BK + PAD) + kv * 8) = reg[i];
        }
    }
};

// outer-contiguous: each thread owns NB blocks of 4 k-rows x 8 outer
// elements; row (k) addresses are evaluated per step.
template <typename T, int R, int BK>
struct TileLoader<T, R, BK, false> {
    static constexpr int KB = 4;
    static constexpr int OG = R / 8;
    static constexpr int NB = (BK / KB) * OG / NT;
    static_assert(NB * NT == (BK / KB) * OG, "tile / thread mismatch");
    u32x4 reg[NB][KB];
    int outer0, outer_max;
    int64_t boff;

    __device__ __forceinline__ void init(const Operand&, int o0, int omax, int64_t b) {
        outer0 = o0; outer_max = omax; boff = b;
    }
    __device__ __forceinline__ void load(const Operand& op, int k0, int K) {
        int tid = threadIdx.x;
#pragma unroll
        for (int b = 0; b < NB; ++b) {
            int blk = tid + b * NT;
            int og = blk % OG, kb = blk / OG;
            int o = outer0 + og * 8;
#pragma unroll
            for (int r = 0; r < KB; ++r) {
                int k = k0 + kb * KB + r;
                u32x4 z = {0u, 0u, 0u, 0u};
                reg[b][r] = z;
                if (k < K && o < outer_max) {
                    int seg = 0;
                    int64_t off = map_off(op.row, (uint32_t)k, op.nseg, &seg);
                    const T* p = reinterpret_cast<const T*>(op.ptr[seg]) + boff + off + o;
                    reg[b][r] = *reinterpret_cast<const u32x4*>(p);
                }
            }
        }
    }
    __device__ __forceinline__ void store(T* lds) {
        int tid = threadIdx.x;
#pragma unroll
        for (int b = 0; b < NB; ++b) {
            int blk = tid + b * NT;
            int og = blk % OG, kb = blk / OG;
            // reg[b][r] holds outer elements og*8 .. og*8+7 of k-row r as 4
            // dwords of 2 x 16 bits; emit, per outer element, its 4 k values.
#pragma unroll
            for (int w = 0; w < 4; ++w) {
                uint32_t r0 = reg[b][0][w], r1 = reg[b][1][w], r2 = reg[b][2][w], r3 = reg[b][3][w];
                u32x2 lo, hi;
                lo[0] = (r0 & 0xFFFFu) | (r1 << 16);
                lo[1] = (r2 & 0xFFFFu) | (r3 << 16);
                hi[0] = (r0 >> 16) | (r1 & 0xFFFF0000u);
                hi[1] = (r2 >> 16) | (r3 & 0xFFFF0000u);
                int o = og * 8 + 2 * w;
                *reinterpret_cast<u32x2*>(lds + o * (BK + PAD) + kb * KB) = lo;
                *reinterpret_cast<u32x2*>(lds + (o + 1) * (BK + PAD) + kb * KB) = hi;
            }
        }
    }
};

template <typename T, int BM, int BN, int BK, bool AKC, bool BKC>
__global__ __launch_bounds__(NT) void gemm_mfma(GemmArgs g) {
    constexpr int WM = BM / 2, WN = BN / 2;
    constexpr int FM = WM / 16, FN = WN / 16;
    constexpr int LDA = BK + PAD;
    constexpr int AS = BM * LDA, BS = BN * LDA;
    constexpr int CLD = BN + 4;
    constexpr int SMEM_AB = 2 * (AS + BS) * (int)sizeof(T);
    constexpr int SMEM_C = BM * CLD * 4;
    constexpr int SMEM = SMEM_AB > SMEM_C ? SMEM_AB : SMEM_C;
    __shared__ __attribute__((aligned(16))) unsigned char smem[SMEM];
    T* As = reinterpret_cast<T*>(smem);
    T* Bs = As + 2 * AS;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int tile = blockIdx.x;
    const int tm = tile / g.tiles_n, tn = tile - tm * g.tiles_n;
    const int m0 = tm * BM, n0 = tn * BN;
    const uint32_t z = blockIdx.y;

    int dummy = 0;
    int64_t aoff = map_off(g.a.batch, z, 1, &dummy);
    int64_t boff = map_off(g.b.batch, z, 1, &dummy);

    TileLoader<T, BM, BK, AKC> la;
    TileLoader<T, BN, BK, BKC> lb;
    la.init(g.a, m0, g.M, aoff);
    lb.init(g.b, n0, g.N, boff);

    floatx4 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

    const int nk = (g.K + BK - 1) / BK;
    la.load(g.a, 0, g.K);
    lb.load(g.b, 0, g.K);
    la.store(As);
    lb.store(Bs);
    __syncthreads();

    typedef typename Mfma<T>::frag frag;
    const int lr = lane & 15, lk = (lane >> 4) * 8;
    for (int s = 0; s < nk; ++s) {
        const int buf = s & 1;
        if (s + 1 < nk) {
            la.load(g.a, (s + 1) * BK, g.K);
            lb.load(g.b, (s + 1) * BK, g.K);
        }
        const T* Ab = As + buf * AS + (wm * WM + lr) * LDA + lk;
        const T* Bb = Bs + buf * BS + (wn * WN + lr) * LDA + lk;
#pragma unroll
        for (int kk = 0; kk < BK; kk += 32) {
            frag af[FM], bf[FN];
#pragma unroll
            for (int i = 0; i < FM; ++i)
                af[i] = __builtin_bit_cast(frag, *reinterpret_cast<const u32x4*>(Ab + i * 16 * LDA + kk));
#pragma unroll
            for (int j = 0; j < FN; ++j)
                bf[j] = __builtin_bit_cast(frag, *reinterpret_cast<const u32x4*>(Bb + j * 16 * LDA + kk));
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j) acc[i][j] = Mfma<T>::run(af[i], bf[j], acc[i][j]);
        }
        if (s + 1 < nk) {
            la.store(As + (buf ^ 1) * AS);
            lb.store(Bs + (buf ^ 1) * BS);
        }
        __syncthreads();
    }

    // ---- epilogue: fp32 tile through LDS, then 8-wide vector stores
    float* Cs = reinterpret_cast<float*>(smem);
    const float alpha = g.c.alpha;
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                int row = wm * WM + i * 16 + (lane >> 4) * 4 + r;
                int col = wn * WN + j * 16 + lr;
                Cs[row * CLD + col] = acc[i][j][r] * alpha;
            }
    __syncthreads();

    const Epilogue& e = g.c;
    int64_t coff = map_off(e.batch, z, 1, &dummy);
    constexpr int NVEC = BM * BN / 8;
    for (int v = tid; v < NVEC; v += NT) {
        int m, n, lm, ln;
        float vals[8];
        if (e.contig_n) {
            lm = v / (BN / 8); ln = (v % (BN / 8)) * 8;
            m = m0 + lm; n = n0 + ln;
            if (m >= g.M || n >= g.N) continue;
#pragma unroll
            for (int q = 0; q < 8; ++q) vals[q] = Cs[lm * CLD + ln + q];
        } else {
            ln = v / (BM / 8); lm = (v % (BM / 8)) * 8;
            m = m0 + lm; n = n0 + ln;
            if (m >= g.M || n >= g.N) continue;
#pragma unroll
            for (int q = 0; q < 8; ++q) vals[q] = Cs[(lm + q) * CLD + ln];
        }
        if (e.bias[0]) {
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                uint32_t idx = e.bias_on_m ? (uint32_t)(e.contig_n ? m : m + q)
                                           : (uint32_t)(e.contig_n ? n + q : n);
                int bseg = 0;
                int64_t bo = map_off(e.bias_map, idx, e.bias_nseg, &bseg);
                vals[q] += to_f(reinterpret_cast<const T*>(e.bias[bseg])[bo]);
            }
        }
        int sm = 0, sn = 0;
        int64_t off = coff + map_off(e.mmap, (uint32_t)m, e.seg_on_m ? e.nseg : 1, &sm) +
                      map_off(e.nmap, (uint32_t)n, e.seg_on_m ? 1 : e.nseg, &sn);
        int seg = e.seg_on_m ? sm : sn;
        if (e.out_f32) {
            float* p = reinterpret_cast<float*>(e.ptr[seg]) + off;
            if (e.resid) {
                float rv[8];
                V8<float>::load(reinterpret_cast<const float*>(e.resid) + off, rv);
#pragma unroll
                for (int q = 0; q < 8; ++q) vals[q] += rv[q];
            }
            V8<float>::store(p, vals);
        } else {
            T* p = reinterpret_cast<T*>(e.ptr[seg]) + off;
            if (e.resid) {
                float rv[8];
                V8<T>::load(reinterpret_cast<const T*>(e.resid) + off, rv);
#pragma unroll
                for (int q = 0; q < 8; ++q) vals[q] += rv[q];
            }
            V8<T>::store(p, vals);
        }
    }
}

// ------------------------------------------------------------ fp32 path
// One output element per thread, operands read through the same maps.
__device__ __forceinline__ float op_elem(const Operand& op, int64_t boff, int outer, int k) {
    int seg = 0;
    if (op.kcontig) {
        int64_t off = map_off(op.row, (uint32_t)outer, op.nseg, &seg);
        return reinterpret_cast<const float*>(op.ptr[seg])[boff + off + k];
    }
    int64_t off = map_off(op.row, (uint32_t)k, op.nseg, &seg);
    return reinterpret_cast<const float*>(op.ptr[seg])[boff + off + outer];
}

__global__ __launch_bounds__(256) void gemm_f32(GemmArgs g) {
    const int n = blockIdx.x * 16 + (threadIdx.x & 15);
    const int m = (blockIdx.y % g.tiles_m) * 16 + (threadIdx.x >> 4);
    const uint32_t z = blockIdx.y / g.tiles_m;
    if (m >= g.M || n >= g.N) return;
    int dummy = 0;
    int64_t aoff = map_off(g.a.batch, z, 1, &dummy);
    int64_t boff = map_off(g.b.batch, z, 1, &dummy);
    float acc = 0.f;
    for (int k = 0; k < g.K; ++k) acc = fmaf(op_elem(g.a, aoff, m, k), op_elem(g.b, boff, n, k), acc);
    const Epilogue& e = g.c;
    float v = acc * e.alpha;
    if (e.bias[0]) {
        int bseg = 0;
        int64_t bo = map_off(e.bias_map, (uint32_t)(e.bias_on_m ? m : n), e.bias_nseg, &bseg);
        v += reinterpret_cast<const float*>(e.bias[bseg])[bo];
    }
    int sm = 0, sn = 0;
    int64_t off = map_off(e.batch, z, 1, &dummy) + map_off(e.mmap, (uint32_t)m, e.seg_on_m ? e.nseg : 1, &sm) +
                  map_off(e.nmap, (uint32_t)n, e.seg_on_m ? 1 : e.nseg, &sn);
    int seg = e.seg_on_m ? sm : sn;
    if (e.resid) v += reinterpret_cast<const float*>(e.resid)[off];
    reinterpret_cast<float*>(e.ptr[seg])[off] = v;
}

template <typename T, int BM, int BN, int BK>
int launch_t(GemmArgs g, hipStream_t st) {
    g.tiles_m = (g.M + BM - 1) / BM;
    g.tiles_n = (g.N + BN - 1) / BN;
    dim3 grid(g.tiles_m * g.tiles_n, g.batch);
    if (g.a.kcontig && g.b.kcontig)
        hipLaunchKernelGGL((gemm_mfma<T, BM, BN, BK, true, true>), grid, dim3(NT), 0, st, g);
    else if (g.a.kcontig)
        hipLaunchKernelGGL((gemm_mfma<T, BM, BN, BK, true, false>), grid, dim3(NT), 0, st, g);
    else if (g.b.kcontig)
        hipLaunchKernelGGL((gemm_mfma<T, BM, BN, BK, false, true>), grid, dim3(NT), 0, st, g);
    else
        hipLaunchKernelGGL((gemm_mfma<T, BM, BN, BK, false, false>), grid, dim3(NT), 0, st, g);
    return 0;
}

}  // namespace

int launch_gemm(int dtype, const GemmArgs& args, hipStream_t st) {
    GemmArgs g = args;
    if (g.M <= 0 || g.N <= 0 || g.batch <= 0) return 0;
    if (g.K <= 0) return set_error(DM_ERR_ARG, "contraction with K <= 0");
    if (g.batch > 65535) return set_error(DM_ERR_UNSUPPORTED, "contraction batch above 65535");
    if (dtype == G_F32) {
        g.tiles_m = (g.M + 15) / 16;
        g.tiles_n = (g.N + 15) / 16;
        if ((int64_t)g.tiles_m * g.batch > 65535)
            return set_error(DM_ERR_UNSUPPORTED, "fp32 contraction grid too large");
        dim3 grid(g.tiles_n, g.tiles_m * g.batch);
        hipLaunchKernelGGL(gemm_f32, grid, dim3(256), 0, st, g);
    } else {
        if (g.K % 8 || g.M % 8 || g.N % 8)
            return set_error(DM_ERR_UNSUPPORTED, "contraction sizes must be multiples of 8");
        if (dtype == G_F16) launch_t<half_t, 128, 128, 64>(g, st);
        else launch_t<bf16_t, 128, 128, 64>(g, st);
    }
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return set_error(DM_ERR_DEVICE, "contraction launch: %s", hipGetErrorString(err));
    return 0;
}

}  // namespace dm
