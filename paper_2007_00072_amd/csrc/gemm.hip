// MFMA contraction kernel for gfx950 (fp16 / bf16 storage, fp32
// accumulation) and an fp32 MFMA kernel (v_mfma_f32_32x32x2f32) for float32 layers.
//
// Block tile BM x BN (256x256 down to 128x64), k-step 64, 4 or 8 wave64s in
// a WGM x WGN grid of wave tiles, v_mfma_f32_16x16x32 inner products.
//
// LDS holds both operands as [outer][k] rows of 64 elements (8 chunks of
// 16 bytes).  Chunk c of row r sits at position c ^ ((r >> 1) & 7): the
// 16-byte fragment reads of 16 consecutive rows then cover all 64 banks
// exactly once, and no padding is needed.
//
// A k-contiguous operand is copied to that layout with 16-byte loads; an
// outer-contiguous operand is copied in its own [k][outer] order and its
// fragments are read with the gfx950 LDS transpose read, so every einsum
// layout reaches the MFMAs without a transpose pass.  Global loads run one or
// two k-steps ahead of the MFMAs (one or two register sets, LDS double
// buffer, one barrier per step).
//
// Tiles are numbered so that each of the 8 XCDs gets a contiguous run of
// tile indices, walked in groups of rows for L2 reuse.  A split-K mode
// writes float partial sums that a second kernel adds in a fixed order
// (deterministic), for contractions with few output tiles and a long k.
// The epilogue stages the fp32 tile through LDS in 64-column passes and
// writes 16-byte vectors along whichever output index is contiguous.
#include <algorithm>
#include <mutex>
#include <string.h>
#include <vector>

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

constexpr int BK = 64;  // k per step = 8 chunks of 8 elements

__device__ __forceinline__ int swz(int row, int chunk) { return chunk ^ ((row >> 1) & 7); }

// Barrier for hand-offs through LDS: waits for this thread's LDS accesses
// only.  (__syncthreads would also wait for every outstanding global store,
// which in the epilogue serialises the passes on the store latency.)
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// Pointer of segment `seg` without indexing the kernel-argument array at
// run time (a dynamic index would turn it into a memory load).
template <typename P>
__device__ __forceinline__ P seg_ptr(P const (&p)[3], int seg) {
    return seg == 0 ? p[0] : (seg == 1 ? p[1] : p[2]);
}

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

template <typename T, int R, int NT, bool KC>
struct Loader;

// k-contiguous operand: thread t owns 16-byte chunk (t & 7) of rows
// t/8, t/8 + NT/8, ...; row pointers are fixed for the whole k loop.  Rows
// past the operand's end read its first row and are zeroed by select, and
// k past the end reads k = 0, so every load is unconditional.
template <typename T, int R, int NT>
struct Loader<T, R, NT, true> {
    static constexpr int NV = R * 8 / NT;
    static_assert(NV >= 1 && NV * NT == R * 8, "tile / thread mismatch");
    typedef u32x4 Regs[NV];
    const T* rowp[NV];
    uint32_t valid;  // bit i: row i in range

    __device__ __forceinline__ void init(const Operand& op, int o0, int omax, int64_t boff) {
        const int tid = threadIdx.x;
        valid = 0;
        int seg0 = 0;
        const int64_t off0 = map_off(op.row, (uint32_t)(o0 < omax ? o0 : 0), op.nseg, &seg0);
        const T* first = reinterpret_cast<const T*>(seg_ptr(op.ptr, seg0)) + boff + off0;
#pragma unroll
        for (int i = 0; i < NV; ++i) {
            const int o = o0 + (tid >> 3) + i * (NT / 8);
            rowp[i] = first;
            if (o < omax) {
                int seg = 0;
                const int64_t off = map_off(op.row, (uint32_t)o, op.nseg, &seg);
                rowp[i] = reinterpret_cast<const T*>(seg_ptr(op.ptr, seg)) + boff + off;
                valid |= 1u << i;
            }
        }
    }
    // Loads never consume their data here (a select on it would make the
    // load wait at once); out-of-range lanes are zeroed when stored.
    __device__ __forceinline__ void load(const Operand&, int k0, int kend, Regs& reg) const {
        const int k = k0 + (threadIdx.x & 7) * 8;
        const int kk = k < kend ? k : 0;
#pragma unroll
        for (int i = 0; i < NV; ++i) reg[i] = *reinterpret_cast<const u32x4*>(rowp[i] + kk);
    }
    // fragment of outer rows ob .. ob+15, k = kk .. kk+31 of this LDS stage:
    // lane l reads row ob + (l & 15), chunk kk/8 + l/16 (one 16-byte read;
    // 16 consecutive rows cover all 64 banks once under the swizzle)
    __device__ __forceinline__ u32x4 frag(const T* lds, int ob, int kk, int lane) const {
        const int r = ob + (lane & 15);
        const int c = (kk >> 3) + (lane >> 4);
        return *reinterpret_cast<const u32x4*>(lds + r * BK + swz(r, c) * 8);
    }
    __device__ __forceinline__ void store(T* lds, const Regs& reg, int k0, int kend) const {
        const int tid = threadIdx.x, c = tid & 7;
        const bool kin = k0 + c * 8 < kend;
#pragma unroll
        for (int i = 0; i < NV; ++i) {
            const int r = (tid >> 3) + i * (NT / 8);
            const u32x4 z = {0u, 0u, 0u, 0u};
            const bool ok = kin && ((valid >> i) & 1u);
            *reinterpret_cast<u32x4*>(lds + r * BK + swz(r, c) * 8) = ok ? reg[i] : z;
        }
    }
};

// outer-contiguous operand: LDS keeps its natural [k][outer] order (rows
// of R elements, 16-byte chunk c of row r at c ^ (2 * (r & 3))), filled by
// plain 16-byte copies.  MFMA fragments are read with the gfx950 transpose
// read ds_read_b64_tr_b16: within a group of 16 lanes, lane i receives
// element i % 4 of the 8-byte pieces addressed by lanes i/4 + 4j, j = 0..3.
// Lane s of group g addresses row k0 + 8g + s/4 (+4 for the second read),
// outer elements 4(s % 4) .. +3, and so receives outer element s at k
// values 8g .. 8g+7: exactly the k-contiguous fragment layout.
template <typename T, int R, int NT>
struct Loader<T, R, NT, false> {
    static constexpr int CPR = R / 8;  // chunks per k-row
    static constexpr int NV = BK * CPR / NT;
    static_assert(NV >= 1 && NV * NT == BK * CPR && CPR >= 8, "tile / thread mismatch");
    typedef u32x4 Regs[NV];
    int o0, omax;
    int64_t boff;

    __device__ __forceinline__ void init(const Operand&, int o0_, int omax_, int64_t b) {
        o0 = o0_; omax = omax_; boff = b;
    }
    __device__ __forceinline__ void load(const Operand& op, int k0, int kend, Regs& reg) const {
#pragma unroll
        for (int i = 0; i < NV; ++i) {
            const int v = threadIdx.x + i * NT;
            const int kr = v / CPR, c = v % CPR;
            const int k = k0 + kr, o = o0 + c * 8;
            const bool in = k < kend && o < omax;
            int seg = 0;
            const int64_t off = map_off(op.row, (uint32_t)(in ? k : 0), op.nseg, &seg);
            reg[i] = *reinterpret_cast<const u32x4*>(reinterpret_cast<const T*>(seg_ptr(op.ptr, seg)) + boff + off +
                                                     (in ? o : 0));
        }
    }
    __device__ __forceinline__ void store(T* lds, const Regs& reg, int k0, int kend) const {
#pragma unroll
        for (int i = 0; i < NV; ++i) {
            const int v = threadIdx.x + i * NT;
            const int kr = v / CPR, c = v % CPR;
            const bool in = k0 + kr < kend && o0 + c * 8 < omax;
            const u32x4 z = {0u, 0u, 0u, 0u};
            *reinterpret_cast<u32x4*>(lds + kr * R + ((c ^ (2 * (kr & 3))) * 8)) = in ? reg[i] : z;
        }
    }
    // fragment of outer rows ob .. ob+15, k = kk .. kk+31 of this LDS stage
    __device__ __forceinline__ u32x4 frag(const T* lds, int ob, int kk, int lane) const {
        typedef short s4 __attribute__((ext_vector_type(4)));
        typedef __attribute__((address_space(3))) s4 lds_s4;
        const int g = lane >> 4, sl = lane & 15;
        const int r = kk + 8 * g + (sl >> 2);
        const int c = (ob >> 3) + ((sl & 3) >> 1);
        const T* p = lds + r * R + ((c ^ (2 * (sl >> 2))) * 8) + (sl & 1) * 4;
        const s4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4*)p);
        const s4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4*)(p + 4 * R));
        u32x4 out;
        out[0] = (uint16_t)lo[0] | ((uint32_t)(uint16_t)lo[1] << 16);
        out[1] = (uint16_t)lo[2] | ((uint32_t)(uint16_t)lo[3] << 16);
        out[2] = (uint16_t)hi[0] | ((uint32_t)(uint16_t)hi[1] << 16);
        out[3] = (uint16_t)hi[2] | ((uint32_t)(uint16_t)hi[3] << 16);
        return out;
    }
};

// ------------------------------------------------------------------ epilogue
// Stores 8 outputs (along n if contig_n, else along m) starting at (m, n)
// of batch z: alpha already applied; adds bias and resid, converts, maps.
template <typename T>
__device__ __forceinline__ void store_vec(const GemmArgs& g, int64_t coff, int m, int n, float vals[8]) {
    const Epilogue& e = g.c;
    if (e.bias[0]) {
        // The 8 outputs share one bias index when the bias runs along the
        // other output index; along the contiguous index they are 8
        // consecutive indices, which stay inside one digit of the bias map
        // (vectors start at multiples of 8 and the launcher checks that the
        // map's lowest radix is a multiple of 8), so one map evaluation and
        // a stride give all of them.
        const bool along = (e.bias_on_m != 0) == (e.contig_n == 0);
        const uint32_t idx = (uint32_t)(e.bias_on_m ? m : n);
        int bseg = 0;
        const int64_t bo = map_off(e.bias_map, idx, e.bias_nseg, &bseg);
        const T* bp = reinterpret_cast<const T*>(seg_ptr(e.bias, bseg)) + bo;
        if (along) {
#pragma unroll
            for (int q = 0; q < 8; ++q) vals[q] += to_f(bp[(int64_t)q * e.bias_map.s0]);
        } else {
            const float bv = to_f(bp[0]);
#pragma unroll
            for (int q = 0; q < 8; ++q) vals[q] += bv;
        }
    }
    int sm = 0, sn = 0;
    const int64_t off = coff + map_off(e.mmap, (uint32_t)m, e.seg_on_m ? e.nseg : 1, &sm) +
                        map_off(e.nmap, (uint32_t)n, e.seg_on_m ? 1 : e.nseg, &sn);
    const int seg = e.seg_on_m ? sm : sn;
    if (e.out_f32) {
        if (e.resid) {
            float rv[8];
            V8<float>::load(reinterpret_cast<const float*>(e.resid) + off, rv);
#pragma unroll
            for (int q = 0; q < 8; ++q) vals[q] += rv[q];
        }
        V8<float>::store(reinterpret_cast<float*>(seg_ptr(e.ptr, seg)) + off, vals);
    } else {
        if (e.resid) {
            float rv[8];
            V8<T>::load(reinterpret_cast<const T*>(e.resid) + off, rv);
#pragma unroll
            for (int q = 0; q < 8; ++q) vals[q] += rv[q];
        }
        V8<T>::store(reinterpret_cast<T*>(seg_ptr(e.ptr, seg)) + off, vals);
    }
}

// Writes one 64-column pass of the output tile, staged in LDS as fp32 rows
// of 68 floats: 16-byte stores along whichever output index is contiguous
// (or float partial sums to the split workspace).
template <typename T, int BM, int NT>
__device__ __forceinline__ void store_pass(const GemmArgs& g, const float* Cs, int m0, int n0, uint32_t z, int sidx,
                                           bool partial, int64_t coff, bool contig_n) {
    constexpr int PW = 64, CLD = PW + 4;
    constexpr int NVEC = BM * PW / 8;
    for (int v = threadIdx.x; v < NVEC; v += NT) {
        int m, n, lm, ln;
        float vals[8];
        if (contig_n) {
            lm = v / (PW / 8); ln = (v % (PW / 8)) * 8;
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
        if (partial) {
            float* dst = g.split_ws + (((int64_t)sidx * g.batch + z) * g.M + m) * (int64_t)g.N + n;
            V8<float>::store(dst, vals);
        } else {
            store_vec<T>(g, coff, m, n, vals);
        }
    }
}

// Store pass for affine outputs (one pointer, unit stride along the
// contiguous index, bias along either index): residual and bias loads for
// all of a thread's vectors are issued before its stores.
template <typename T, int BM, int NT>
__device__ __forceinline__ void store_pass_affine(const GemmArgs& g, const float* Cs, int m0, int n0, int64_t coff,
                                                  bool contig_n) {
    constexpr int PW = 64, CLD = PW + 4;
    constexpr int NVEC = BM * PW / 8;
    constexpr int VPT = NVEC / NT;
    static_assert(VPT * NT == NVEC, "pass / thread mismatch");
    const Epilogue& e = g.c;
    const int tid = threadIdx.x;
    int lm[VPT], ln[VPT];
    bool ok[VPT];
    int64_t off[VPT];
#pragma unroll
    for (int i = 0; i < VPT; ++i) {
        const int v = tid + i * NT;
        if (contig_n) { lm[i] = v / (PW / 8); ln[i] = (v % (PW / 8)) * 8; }
        else { ln[i] = v / (BM / 8); lm[i] = (v % (BM / 8)) * 8; }
        const int m = m0 + lm[i], n = n0 + ln[i];
        ok[i] = m < g.M && n < g.N;
        off[i] = coff + (contig_n ? (int64_t)m * g.ldc + n : (int64_t)m + (int64_t)n * g.ldc);
    }
    float add[VPT][8];
#pragma unroll
    for (int i = 0; i < VPT; ++i)
#pragma unroll
        for (int q = 0; q < 8; ++q) add[i][q] = 0.f;
    if (g.bias_mode == 1) {
        const T* b = reinterpret_cast<const T*>(e.bias[0]);
#pragma unroll
        for (int i = 0; i < VPT; ++i)
            if (ok[i]) V8<T>::load(b + (contig_n ? n0 + ln[i] : m0 + lm[i]), add[i]);
    } else if (g.bias_mode == 2) {
        const T* b = reinterpret_cast<const T*>(e.bias[0]);
#pragma unroll
        for (int i = 0; i < VPT; ++i)
            if (ok[i]) {
                const float bv = to_f(b[contig_n ? m0 + lm[i] : n0 + ln[i]]);
#pragma unroll
                for (int q = 0; q < 8; ++q) add[i][q] = bv;
            }
    }
    if (e.resid) {
#pragma unroll
        for (int i = 0; i < VPT; ++i)
            if (ok[i]) {
                float rv[8];
                if (e.out_f32) V8<float>::load(reinterpret_cast<const float*>(e.resid) + off[i], rv);
                else V8<T>::load(reinterpret_cast<const T*>(e.resid) + off[i], rv);
#pragma unroll
                for (int q = 0; q < 8; ++q) add[i][q] += rv[q];
            }
    }
#pragma unroll
    for (int i = 0; i < VPT; ++i) {
        float vals[8];
        if (contig_n) {
#pragma unroll
            for (int q = 0; q < 8; ++q) vals[q] = Cs[lm[i] * CLD + ln[i] + q] + add[i][q];
        } else {
#pragma unroll
            for (int q = 0; q < 8; ++q) vals[q] = Cs[(lm[i] + q) * CLD + ln[i]] + add[i][q];
        }
        if (!ok[i]) continue;
        if (e.out_f32) V8<float>::store(reinterpret_cast<float*>(e.ptr[0]) + off[i], vals);
        else V8<T>::store(reinterpret_cast<T*>(e.ptr[0]) + off[i], vals);
    }
}

// ------------------------------------------------------------------ epilogue
// 64-column passes of the fp32 tile through LDS (smem, at least
// BM * 68 floats), then 16-byte stores along the contiguous output index;
// with split k, float partial sums go to the split workspace instead.
template <typename T, int BM, int BN, int WGM, int WGN>
__device__ __forceinline__ void epilogue(const GemmArgs& g, const floatx4 (&acc)[BM / WGM / 16][BN / WGN / 16],
                                         unsigned char* smem, int m0, int n0, uint32_t z, int sidx, int splits) {
    constexpr int NT = 64 * WGM * WGN;
    constexpr int WM = BM / WGM, WN = BN / WGN;
    constexpr int FM = WM / 16, FN = WN / 16;
    constexpr int PW = 64, CLD = PW + 4;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave / WGN, wn = wave % WGN;
    const int lr = lane & 15, lc = lane >> 4;
    int dummy = 0;
    float* Cs = reinterpret_cast<float*>(smem);
    const bool partial = splits > 1;
    const float alpha = partial ? 1.0f : g.c.alpha;
    const int64_t coff = partial ? 0 : map_off(g.c.batch, z, 1, &dummy);
    const bool contig_n = partial ? true : g.c.contig_n != 0;
#pragma unroll
    for (int p = 0; p < BN / PW; ++p) {
#pragma unroll
        for (int j = 0; j < FN; ++j) {
            const int col = wn * WN + j * 16;
            if (col < p * PW || col >= (p + 1) * PW) continue;
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int row = wm * WM + i * 16 + lc * 4 + r;
                    Cs[row * CLD + col - p * PW + lr] = acc[i][j][r] * alpha;
                }
        }
        lds_barrier();
        if (g.affine && !partial) store_pass_affine<T, BM, NT>(g, Cs, m0, n0 + p * PW, coff, contig_n);
        else store_pass<T, BM, NT>(g, Cs, m0, n0 + p * PW, z, sidx, partial, coff, contig_n);
        lds_barrier();
    }
}

// Block -> (tile, batch index).  Workgroups reach the 8 XCDs round-robin
// by linear id (x fastest); linear ids are renumbered so that each XCD's
// share is one contiguous run of (batch, tile) indices: the tiles of one
// batch entry, and neighbouring tiles of a large contraction, then share
// that XCD's L2.  Within a batch entry tiles go in groups of GM tile rows
// (column-major inside a group) so concurrently running tiles reuse both
// operand panels.
__device__ __forceinline__ int xcd_order(int lid, int total) {
    return (total & 7) == 0 ? (lid & 7) * (total >> 3) + (lid >> 3) : lid;
}
__device__ __forceinline__ void tile_in(int t, int tiles_m, int tiles_n, int& tm, int& tn) {
    constexpr int GM = 4;
    const int per_group = GM * tiles_n;
    const int grp = t / per_group;
    const int first = grp * GM;
    const int gm = min(tiles_m - first, GM);
    const int r = t - grp * per_group;
    tm = first + r % gm;
    tn = r / gm;
}
__device__ __forceinline__ void tile_of(int tiles_m, int tiles_n, int& tm, int& tn, int& by) {
    const int nt = tiles_m * tiles_n;
    const int lid = xcd_order((int)blockIdx.y * nt + (int)blockIdx.x, nt * (int)gridDim.y);
    by = lid / nt;
    tile_in(lid - by * nt, tiles_m, tiles_n, tm, tn);
}

template <typename T, int BM, int BN, int WGM, int WGN, int DEPTH, bool AKC, bool BKC>
__global__ __launch_bounds__(64 * WGM * WGN) void gemm_mfma(GemmArgs g) {
    constexpr int NT = 64 * WGM * WGN;
    constexpr int WM = BM / WGM, WN = BN / WGN;
    constexpr int FM = WM / 16, FN = WN / 16;
    constexpr int AS = BM * BK, BS = BN * BK;
    constexpr int SMEM_AB = 2 * (AS + BS) * (int)sizeof(T);
    constexpr int PW = 64, CLD = PW + 4;
    static_assert(BM * CLD * 4 <= SMEM_AB, "epilogue staging does not fit");
    static_assert(WM % 16 == 0 && WN % 16 == 0 && BN % PW == 0, "bad tile");
    __shared__ __attribute__((aligned(16))) unsigned char smem[SMEM_AB];
    T* As = reinterpret_cast<T*>(smem);
    T* Bs = As + 2 * AS;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave / WGN, wn = wave % WGN;
    int tm, tn;
    int by;
    tile_of(g.tiles_m, g.tiles_n, tm, tn, by);
    const int m0 = tm * BM, n0 = tn * BN;
    const int splits = g.splits > 1 ? g.splits : 1;
    const uint32_t z = (uint32_t)by / splits;
    const int sidx = by - (int)z * splits;
    const int kb = splits > 1 ? sidx * g.kper : 0;
    const int ke = splits > 1 ? min(g.K, kb + g.kper) : g.K;

    int dummy = 0;
    const int64_t aoff = map_off(g.a.batch, z, 1, &dummy);
    const int64_t boff = map_off(g.b.batch, z, 1, &dummy);

    Loader<T, BM, NT, AKC> la;
    Loader<T, BN, NT, BKC> lb;
    la.init(g.a, m0, g.M, aoff);
    lb.init(g.b, n0, g.N, boff);

    floatx4 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

    typedef typename Mfma<T>::frag frag;
    const int lr = lane & 15, lc = lane >> 4;
    auto compute = [&](int buf) {
        const T* Ab = As + buf * AS;
        const T* Bb = Bs + buf * BS;
#pragma unroll
        for (int kk = 0; kk < BK; kk += 32) {
            frag af[FM], bf[FN];
#pragma unroll
            for (int i = 0; i < FM; ++i) af[i] = __builtin_bit_cast(frag, la.frag(Ab, wm * WM + i * 16, kk, lane));
#pragma unroll
            for (int j = 0; j < FN; ++j) bf[j] = __builtin_bit_cast(frag, lb.frag(Bb, wn * WN + j * 16, kk, lane));
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j) acc[i][j] = Mfma<T>::run(af[i], bf[j], acc[i][j]);
        }
    };

    const int nk = ke > kb ? (ke - kb + BK - 1) / BK : 0;
    if constexpr (DEPTH == 2) {
        // Two register sets hold the k-steps in flight: step s+1 was
        // requested one step ago and is written to LDS at the end of step
        // s, while step s+2 is requested at the start of step s (loop
        // unrolled by two so the sets have fixed registers).
        typename Loader<T, BM, NT, AKC>::Regs ra0, ra1;
        typename Loader<T, BN, NT, BKC>::Regs rb0, rb1;
        if (nk > 0) {
            la.load(g.a, kb, ke, ra0);
            lb.load(g.b, kb, ke, rb0);
            la.store(As, ra0, kb, ke);
            lb.store(Bs, rb0, kb, ke);
            if (nk > 1) {
                la.load(g.a, kb + BK, ke, ra1);
                lb.load(g.b, kb + BK, ke, rb1);
            }
        }
        __syncthreads();
        for (int s = 0; s < nk; s += 2) {
            // even step: LDS buffer 0 holds step s, set 1 holds step s+1
            if (s + 2 < nk) {
                la.load(g.a, kb + (s + 2) * BK, ke, ra0);
                lb.load(g.b, kb + (s + 2) * BK, ke, rb0);
            }
            compute(0);
            if (s + 1 < nk) {
                la.store(As + AS, ra1, kb + (s + 1) * BK, ke);
                lb.store(Bs + BS, rb1, kb + (s + 1) * BK, ke);
            }
            __syncthreads();
            if (s + 1 >= nk) break;
            // odd step: LDS buffer 1 holds step s+1, set 0 holds step s+2
            if (s + 3 < nk) {
                la.load(g.a, kb + (s + 3) * BK, ke, ra1);
                lb.load(g.b, kb + (s + 3) * BK, ke, rb1);
            }
            compute(1);
            if (s + 2 < nk) {
                la.store(As, ra0, kb + (s + 2) * BK, ke);
                lb.store(Bs, rb0, kb + (s + 2) * BK, ke);
            }
            __syncthreads();
        }
    } else {
        // One register set: step s+1 is requested at the start of step s.
        typename Loader<T, BM, NT, AKC>::Regs ra;
        typename Loader<T, BN, NT, BKC>::Regs rb;
        if (nk > 0) {
            la.load(g.a, kb, ke, ra);
            lb.load(g.b, kb, ke, rb);
            la.store(As, ra, kb, ke);
            lb.store(Bs, rb, kb, ke);
        }
        __syncthreads();
        for (int s = 0; s < nk; ++s) {
            const int buf = s & 1;
            if (s + 1 < nk) {
                la.load(g.a, kb + (s + 1) * BK, ke, ra);
                lb.load(g.b, kb + (s + 1) * BK, ke, rb);
            }
            compute(buf);
            if (s + 1 < nk) {
                la.store(As + (buf ^ 1) * AS, ra, kb + (s + 1) * BK, ke);
                lb.store(Bs + (buf ^ 1) * BS, rb, kb + (s + 1) * BK, ke);
            }
            __syncthreads();
        }
    }

    epilogue<T, BM, BN, WGM, WGN>(g, acc, smem, m0, n0, z, sidx, splits);
}


// ------------------------------------------------------ asynchronous variant
// Same LDS layouts and fragment reads as gemm_mfma, but operands move from
// global memory straight into LDS (global_load_lds_dwordx4: lane l of a
// wave writes 16 bytes at M0 + 16 l), through a ring of three LDS stages
// with two k-steps in flight.  The copies are issued from inline assembly
// so that the compiler neither waits for them early nor reorders LDS
// accesses around them; each thread waits for its own copies of a stage
// with s_waitcnt vmcnt before the barrier that publishes the stage.
__device__ __attribute__((aligned(16))) uint32_t g_zero16[4] = {0u, 0u, 0u, 0u};

__device__ __forceinline__ void lds_dma16(const void* src, uint32_t lds_byte) {
    asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(src),
                 "s"(__builtin_amdgcn_readfirstlane(lds_byte))
                 : "memory", "m0");
}

template <int N>
__device__ __forceinline__ void wait_vm() {
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

__device__ __forceinline__ uint32_t lds_addr(const void* p) {
    return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) char*)p;
}

template <typename T, int R, int NT, bool KC, int SW = 2>
struct Dma;

// k-contiguous: slot q = i*NT + tid of a stage holds row q/8, physical
// chunk q%8, i.e. logical chunk (q%8) ^ ((row>>1)&7).
template <typename T, int R, int NT, int SW>
struct Dma<T, R, NT, true, SW> {
    static constexpr int NV = R * 8 / NT;
    static_assert(NV >= 1 && NV * NT == R * 8, "tile / thread mismatch");
    const T* src[NV];  // element pointer of the thread's chunk at k = 0
    int cofs[NV];      // k offset of that chunk

    __device__ __forceinline__ void init(const Operand& op, int o0, int omax, int64_t boff) {
        const int tid = threadIdx.x;
#pragma unroll
        for (int i = 0; i < NV; ++i) {
            const int q = i * NT + tid, r = q >> 3, c = (q & 7) ^ ((r >> 1) & 7);
            const int o = o0 + r < omax ? o0 + r : (omax > 0 ? omax - 1 : 0);
            int seg = 0;
            const int64_t off = map_off(op.row, (uint32_t)o, op.nseg, &seg);
            src[i] = reinterpret_cast<const T*>(seg_ptr(op.ptr, seg)) + boff + off;
            cofs[i] = c * 8;
        }
    }
    __device__ __forceinline__ void issue(const Operand&, int k0, int kend, uint32_t stage_lds) const {
        const int w = threadIdx.x >> 6;
#pragma unroll
        for (int i = 0; i < NV; ++i) {
            const int k = k0 + cofs[i];
            const void* p = k < kend ? (const void*)(src[i] + k) : (const void*)g_zero16;
            lds_dma16(p, stage_lds + (uint32_t)(i * NT + w * 64) * 16u);
        }
    }
};

// outer-contiguous: slot q holds k-row q/CPR, physical chunk q%CPR, i.e.
// logical chunk (q%CPR) ^ (SW*(row&3)).
template <typename T, int R, int NT, int SW>
struct Dma<T, R, NT, false, SW> {
    static constexpr int CPR = R / 8;
    static constexpr int NV = 64 * CPR / NT;
    static_assert(NV >= 1 && NV * NT == 64 * CPR && CPR >= 8 && 3 * SW < CPR, "tile / thread mismatch");
    int kr[NV];
    int oofs[NV];
    int64_t boff;

    __device__ __forceinline__ void init(const Operand&, int o0, int omax, int64_t b) {
        const int tid = threadIdx.x;
        boff = b;
#pragma unroll
        for (int i = 0; i < NV; ++i) {
            const int q = i * NT + tid;
            kr[i] = q / CPR;
            const int c = (q % CPR) ^ (SW * (kr[i] & 3));
            const int o = o0 + c * 8;
            oofs[i] = o < omax ? o : 0;
        }
    }
    __device__ __forceinline__ void issue(const Operand& op, int k0, int kend, uint32_t stage_lds) const {
        const int w = threadIdx.x >> 6;
#pragma unroll
        for (int i = 0; i < NV; ++i) {
            // k0 < kend always holds here, so k0 is a valid row for the
            // lanes whose own row is past the end (they read zeros instead)
            const int k = k0 + kr[i];
            const bool in = k < kend;
            int seg = 0;
            const int64_t off = map_off(op.row, (uint32_t)(in ? k : k0), op.nseg, &seg);
            const T* src = reinterpret_cast<const T*>(seg_ptr(op.ptr, seg)) + boff + off + oofs[i];
            lds_dma16(in ? (const void*)src : (const void*)g_zero16, stage_lds + (uint32_t)(i * NT + w * 64) * 16u);
        }
    }
};

template <typename T, int BM, int BN, int WGM, int WGN, bool AKC, bool BKC>
__global__ __launch_bounds__(64 * WGM * WGN) void gemm_dma(GemmArgs g) {
    constexpr int NT = 64 * WGM * WGN;
    constexpr int WM = BM / WGM, WN = BN / WGN;
    constexpr int FM = WM / 16, FN = WN / 16;
    constexpr int AS = BM * BK, BS = BN * BK;       // elements per stage
    constexpr int STAGE = (AS + BS) * (int)sizeof(T);  // bytes per stage
    constexpr int SMEM = 3 * STAGE;
    static_assert(BM * 68 * 4 <= SMEM, "epilogue staging does not fit");
    __shared__ __attribute__((aligned(16))) unsigned char smem[SMEM];
    typedef Dma<T, BM, NT, AKC> DA;
    typedef Dma<T, BN, NT, BKC> DB;
    constexpr int NLOADS = DA::NV + DB::NV;  // copies per thread per stage

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave / WGN, wn = wave % WGN;
    int tm, tn;
    int by;
    tile_of(g.tiles_m, g.tiles_n, tm, tn, by);
    const int m0 = tm * BM, n0 = tn * BN;
    const int splits = g.splits > 1 ? g.splits : 1;
    const uint32_t z = (uint32_t)by / splits;
    const int sidx = by - (int)z * splits;
    const int kb = splits > 1 ? sidx * g.kper : 0;
    const int ke = splits > 1 ? min(g.K, kb + g.kper) : g.K;
    int dummy = 0;
    DA da;
    DB db;
    da.init(g.a, m0, g.M, map_off(g.a.batch, z, 1, &dummy));
    db.init(g.b, n0, g.N, map_off(g.b.batch, z, 1, &dummy));
    // only the fragment readers of the staged loaders are used
    const Loader<T, BM, 64 * WGM * WGN, AKC> fa{};
    const Loader<T, BN, 64 * WGM * WGN, BKC> fb{};
    const uint32_t base = lds_addr(smem);

    floatx4 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

    typedef typename Mfma<T>::frag frag;
    const int nk = ke > kb ? (ke - kb + BK - 1) / BK : 0;
    auto issue = [&](int s) {
        const uint32_t st = base + (uint32_t)((s % 3) * STAGE);
        da.issue(g.a, kb + s * BK, ke, st);
        db.issue(g.b, kb + s * BK, ke, st + (uint32_t)(AS * sizeof(T)));
    };
    if (nk > 0) issue(0);
    if (nk > 1) issue(1);
    for (int s = 0; s < nk; ++s) {
        if (s + 1 < nk) wait_vm<NLOADS>();
        else wait_vm<0>();
        __builtin_amdgcn_s_barrier();
        if (s + 2 < nk) issue(s + 2);
        const T* Ab = reinterpret_cast<const T*>(smem + (s % 3) * STAGE);
        const T* Bb = Ab + AS;
#pragma unroll
        for (int kk = 0; kk < BK; kk += 32) {
            frag af[FM], bf[FN];
#pragma unroll
            for (int i = 0; i < FM; ++i) af[i] = __builtin_bit_cast(frag, fa.frag(Ab, wm * WM + i * 16, kk, lane));
#pragma unroll
            for (int j = 0; j < FN; ++j) bf[j] = __builtin_bit_cast(frag, fb.frag(Bb, wn * WN + j * 16, kk, lane));
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j) acc[i][j] = Mfma<T>::run(af[i], bf[j], acc[i][j]);
        }
    }
    __syncthreads();
    epilogue<T, BM, BN, WGM, WGN>(g, acc, smem, m0, n0, z, sidx, splits);
}

// ------------------------------------------------- 32x32x16 MFMA variant
// v_mfma_f32_32x32x16: lane l holds A row l%32 (B column l%32) at k values
// 8(l/32) .. +7; result element r of lane l is row 8(r/4) + 4(l/32) + r%4,
// column l%32.  This instruction runs at the full MFMA rate with only a few
// independent accumulators, where the 16x16x32 form needs many more.
template <typename T> struct Mfma32;
template <> struct Mfma32<half_t> {
    typedef half8 frag;
    __device__ __forceinline__ static floatx16 run(frag a, frag b, floatx16 c) {
        return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
    }
};
template <> struct Mfma32<bf16_t> {
    typedef bf16x8 frag;
    __device__ __forceinline__ static floatx16 run(frag a, frag b, floatx16 c) {
        return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
    }
};

template <typename T, int R, bool KC>
struct Frag32;

// k-contiguous LDS rows (BK elements, chunks swizzled by swz): lane l reads
// row ob + l%32, chunk kk/8 + l/32.
template <typename T, int R>
struct Frag32<T, R, true> {
    __device__ __forceinline__ static u32x4 read(const T* lds, int ob, int kk, int lane) {
        const int r = ob + (lane & 31);
        const int c = (kk >> 3) + (lane >> 5);
        return *reinterpret_cast<const u32x4*>(lds + r * BK + swz(r, c) * 8);
    }
};

// [k][outer] LDS rows of R elements, chunk c of row r stored at
// c ^ (4 (r & 3)): lanes 16g .. 16g+15 take outer ob + 16 (g % 2) + l%16 at
// k = kk + 8 (g / 2) .. +7 with two transposing reads (the lane pattern of
// ds_read_b64_tr_b16 is described at Loader<T, R, NT, false>).  The four
// k-rows one read touches land on four different 64-byte bank groups.
template <typename T, int R>
struct Frag32<T, R, false> {
    static_assert(R >= 128, "outer tile too narrow for the swizzle");
    __device__ __forceinline__ static u32x4 read(const T* lds, int ob, int kk, int lane) {
        typedef short s4 __attribute__((ext_vector_type(4)));
        typedef __attribute__((address_space(3))) s4 lds_s4;
        const int g = lane >> 4, sl = lane & 15;
        const int r = kk + 8 * (g >> 1) + (sl >> 2);
        const int c = ((ob + 16 * (g & 1)) >> 3) + ((sl & 3) >> 1);
        const T* p = lds + r * R + ((c ^ (4 * (sl >> 2))) * 8) + (sl & 1) * 4;
        const s4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4*)p);
        const s4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4*)(p + 4 * R));
        u32x4 out;
        out[0] = (uint16_t)lo[0] | ((uint32_t)(uint16_t)lo[1] << 16);
        out[1] = (uint16_t)lo[2] | ((uint32_t)(uint16_t)lo[3] << 16);
        out[2] = (uint16_t)hi[0] | ((uint32_t)(uint16_t)hi[1] << 16);
        out[3] = (uint16_t)hi[2] | ((uint32_t)(uint16_t)hi[3] << 16);
        return out;
    }
};

// True when map m is affine over every aligned block of 32 indices (its
// lowest radix is unbounded or a multiple of 32), so offset(x + d) =
// offset(x) + d * s0 and the segment stay fixed for x % 32 == 0, d < 32.
inline bool block32_linear(const IdxMap& m) { return m.r0 == 0 || m.r0 % 32 == 0; }

// Epilogue of the 32x32x16 kernels, straight from the accumulators: no LDS
// staging and no barrier, so each wave stores as soon as its own tile is
// done.  In a 32x32 result, lane l holds column l % 32 at rows 8 (r / 4) +
// 4 (l / 32) + r % 4, r = 0..15: with the output contiguous along n, the
// 32 lanes of a half-wave write 32 consecutive elements of one row (the
// memory system merges them into one run); contiguous along m, each lane
// writes the 4 consecutive rows of one r / 4 group as one 8-byte (16-byte
// for fp32) store.  Output offsets are evaluated once per 32-wide block of
// rows and columns: the launcher keeps contractions whose output maps are
// not affine over such blocks (g.blk32), or that take a residual operand or
// a bias along m, on the 16x16x32 kernels.  Biases are loaded before the
// first store: vector-memory waits count loads and stores together, so a
// load between stores would wait for all of them.  With split k the values
// are float partial sums into the split workspace.
// Stores of one wave's WM x WN tile for one output type and orientation
// (the dispatcher below picks the instance once, so the unrolled stores
// carry no per-element branches).  Per 32-row block i: ubase = uniform
// byte address of row mb (segment on m, batch), per 32x32 block j: the
// lane's column offset; inside the block, rows step by rsb bytes.  M is a
// multiple of 8, so each group of 4 rows is either wholly inside or
// wholly outside.
template <typename OutT, bool CN, int WM, int WN>
__device__ __forceinline__ void store_tile(const GemmArgs& g, const floatx16 (&acc)[WM / 32][WN / 32], int mw,
                                           int nw, int64_t coff, const float (&bn)[WN / 32]) {
    constexpr int FM = WM / 32, FN = WN / 32;
    const int lane = threadIdx.x & 63, c = lane & 31, h = lane >> 5;
    const Epilogue& e = g.c;
    const float alpha = e.alpha;
    const int64_t rs = g.affine ? (CN ? g.ldc : 1) : e.mmap.s0;
    const uint32_t rsb = (uint32_t)(rs * (int64_t)sizeof(OutT));
#pragma unroll
    for (int i = 0; i < FM; ++i) {
        const int mb = mw + i * 32;
        if (mb >= g.M) break;
        int64_t rbase;
        int mseg = 0;
        if (g.affine) rbase = (int64_t)mb * rs;
        else rbase = map_off(e.mmap, (uint32_t)mb, e.seg_on_m ? e.nseg : 1, &mseg);
#pragma unroll
        for (int j = 0; j < FN; ++j) {
            const int n = nw + j * 32 + c;
            int nsg = 0;
            int64_t ncol;
            if (g.affine) ncol = CN ? (int64_t)n : (int64_t)n * g.ldc;
            else ncol = map_off(e.nmap, (uint32_t)(n < g.N ? n : 0), e.seg_on_m ? 1 : e.nseg, &nsg);
            char* pb = reinterpret_cast<char*>(seg_ptr(e.ptr, e.seg_on_m ? mseg : nsg)) +
                       (coff + rbase + ncol) * (int64_t)sizeof(OutT) + (CN ? (uint32_t)(4 * h) * rsb
                                                                          : (uint32_t)(4 * h) * sizeof(OutT));
            const bool col_ok = n < g.N;
#pragma unroll
            for (int rg = 0; rg < 4; ++rg) {
                if (!col_ok || mb + 8 * rg + 4 * h >= g.M) continue;
                float v[4];
#pragma unroll
                for (int k = 0; k < 4; ++k) v[k] = acc[i][j][4 * rg + k] * alpha + bn[j];
                if (CN) {
#pragma unroll
                    for (int k = 0; k < 4; ++k)
                        *reinterpret_cast<OutT*>(pb + (uint32_t)(8 * rg + k) * rsb) = from_f<OutT>(v[k]);
                } else {
                    char* q = pb + 8 * rg * (int)sizeof(OutT);
                    if constexpr (sizeof(OutT) == 4) {
                        floatx4 o = {v[0], v[1], v[2], v[3]};
                        *reinterpret_cast<floatx4*>(q) = o;
                    } else {
                        OutT o4[4];
#pragma unroll
                        for (int k = 0; k < 4; ++k) o4[k] = from_f<OutT>(v[k]);
                        *reinterpret_cast<u32x2*>(q) = __builtin_bit_cast(u32x2, o4);
                    }
                }
            }
        }
    }
}

template <typename T, int WM, int WN>
__device__ __forceinline__ void epilogue_direct(const GemmArgs& g, const floatx16 (&acc)[WM / 32][WN / 32],
                                                int mw, int nw, uint32_t z, int sidx, int splits) {
    constexpr int FM = WM / 32, FN = WN / 32;
    const int lane = threadIdx.x & 63, c = lane & 31, h = lane >> 5;
    const Epilogue& e = g.c;
    if (splits > 1) {
        float* base = g.split_ws + ((int64_t)sidx * g.batch + z) * g.M * (int64_t)g.N;
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
            for (int j = 0; j < FN; ++j) {
                const int n = nw + j * 32 + c;
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int m = mw + i * 32 + 8 * (r >> 2) + 4 * h + (r & 3);
                    if (m < g.M && n < g.N) base[(int64_t)m * g.N + n] = acc[i][j][r];
                }
            }
        return;
    }
    int dummy = 0;
    const int64_t coff = map_off(e.batch, z, 1, &dummy);
    // bias along n (the launcher keeps bias-along-m contractions on the
    // 16x16x32 kernels): one value per 32-column block, loaded before any store
    float bn[FN];
#pragma unroll
    for (int j = 0; j < FN; ++j) {
        bn[j] = 0.f;
        if (e.bias[0]) {
            const int n = nw + j * 32 + c;
            int bseg = 0;
            const int64_t bo = map_off(e.bias_map, (uint32_t)(n < g.N ? n : 0), e.bias_nseg, &bseg);
            bn[j] = to_f(reinterpret_cast<const T*>(seg_ptr(e.bias, bseg))[bo]);
        }
    }
    if (e.contig_n) {
        if (e.out_f32) store_tile<float, true, WM, WN>(g, acc, mw, nw, coff, bn);
        else store_tile<T, true, WM, WN>(g, acc, mw, nw, coff, bn);
    } else {
        if (e.out_f32) store_tile<float, false, WM, WN>(g, acc, mw, nw, coff, bn);
        else store_tile<T, false, WM, WN>(g, acc, mw, nw, coff, bn);
    }
}

// Waits until at most `after` stages of this thread's copies are still in
// flight (the copies of one stage are NL instructions).
template <int NL, int STAGES>
__device__ __forceinline__ void wait_stages(int after) {
    if (STAGES >= 4 && after >= 2) wait_vm<2 * NL>();
    else if (STAGES >= 3 && after >= 1) wait_vm<NL>();
    else wait_vm<0>();
}

// Asynchronous-copy contraction on 32x32x16 MFMAs: a ring of STAGES LDS
// stages (BK = 64 each) with STAGES - 1 k-steps in flight; inside a stage
// the fragments of the next 16-wide k slice are read while the current
// slice's MFMAs run.
template <typename T, int BM, int BN, int WGM, int WGN, int STAGES, bool AKC, bool BKC>
__global__ __launch_bounds__(64 * WGM * WGN) void gemm_x32(GemmArgs g) {
    constexpr int NT = 64 * WGM * WGN;
    constexpr int WM = BM / WGM, WN = BN / WGN;
    constexpr int FM = WM / 32, FN = WN / 32;
    constexpr int AS = BM * BK, BS = BN * BK;
    constexpr int STAGE = (AS + BS) * (int)sizeof(T);
    constexpr int RING = STAGES * STAGE;
    constexpr int SMEM = RING > BM * 68 * 4 ? RING : BM * 68 * 4;
    static_assert(STAGES >= 2 && STAGES <= 4 && FM >= 1 && FN >= 1, "configuration");
    static_assert(WGM * WGN * 32 * (WN + 8) * 4 <= SMEM, "epilogue strips do not fit");
    __shared__ __attribute__((aligned(16))) unsigned char smem[SMEM];
    typedef Dma<T, BM, NT, AKC, 4> DA;
    typedef Dma<T, BN, NT, BKC, 4> DB;
    constexpr int NLOADS = DA::NV + DB::NV;
    typedef typename Mfma32<T>::frag frag;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave / WGN, wn = wave % WGN;
    int tm, tn;
    int by;
    tile_of(g.tiles_m, g.tiles_n, tm, tn, by);
    const int m0 = tm * BM, n0 = tn * BN;
    const int splits = g.splits > 1 ? g.splits : 1;
    const uint32_t z = (uint32_t)by / splits;
    const int sidx = by - (int)z * splits;
    const int kb = splits > 1 ? sidx * g.kper : 0;
    const int ke = splits > 1 ? min(g.K, kb + g.kper) : g.K;
    int dummy = 0;
    DA da;
    DB db;
    da.init(g.a, m0, g.M, map_off(g.a.batch, z, 1, &dummy));
    db.init(g.b, n0, g.N, map_off(g.b.batch, z, 1, &dummy));
    const uint32_t base = lds_addr(smem);

    floatx16 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    const int nk = ke > kb ? (ke - kb + BK - 1) / BK : 0;
    auto issue = [&](int s) {
        const uint32_t st = base + (uint32_t)((s % STAGES) * STAGE);
        da.issue(g.a, kb + s * BK, ke, st);
        db.issue(g.b, kb + s * BK, ke, st + (uint32_t)(AS * sizeof(T)));
    };
#pragma unroll
    for (int s = 0; s < STAGES - 1; ++s)
        if (s < nk) issue(s);
    for (int s = 0; s < nk; ++s) {
        const int after = min(STAGES - 2, nk - 1 - s);
        wait_stages<NLOADS, STAGES>(after);
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
        if (s + STAGES - 1 < nk) issue(s + STAGES - 1);
        const T* Ab = reinterpret_cast<const T*>(smem + (s % STAGES) * STAGE);
        const T* Bb = Ab + AS;
        frag af[2][FM], bf[2][FN];
#pragma unroll
        for (int i = 0; i < FM; ++i) af[0][i] = __builtin_bit_cast(frag, Frag32<T, BM, AKC>::read(Ab, wm * WM + i * 32, 0, lane));
#pragma unroll
        for (int j = 0; j < FN; ++j) bf[0][j] = __builtin_bit_cast(frag, Frag32<T, BN, BKC>::read(Bb, wn * WN + j * 32, 0, lane));
#pragma unroll
        for (int q = 0; q < BK / 16; ++q) {
            const int cur = q & 1, nxt = cur ^ 1;
            if (q + 1 < BK / 16) {
#pragma unroll
                for (int i = 0; i < FM; ++i)
                    af[nxt][i] = __builtin_bit_cast(frag, Frag32<T, BM, AKC>::read(Ab, wm * WM + i * 32, (q + 1) * 16, lane));
#pragma unroll
                for (int j = 0; j < FN; ++j)
                    bf[nxt][j] = __builtin_bit_cast(frag, Frag32<T, BN, BKC>::read(Bb, wn * WN + j * 32, (q + 1) * 16, lane));
            }
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j) acc[i][j] = Mfma32<T>::run(af[cur][i], bf[cur][j], acc[i][j]);
        }
    }
    epilogue_direct<T, WM, WN>(g, acc, m0 + wm * WM, n0 + wn * WN, z, sidx, splits);
}

// -------------------------------------------- 256x256 kernel, 4 waves
// Each wave owns a 128x128 quarter of the block tile (4x4 tiles of
// 32x32x16 MFMAs, 256 accumulators), which halves the LDS fragment traffic
// per MFMA against 128x64 wave tiles.  k-step 32, a ring of four LDS stages
// fed by asynchronous copies three k-steps ahead.  Fragments of the next
// 16-wide k slice are read while the current slice's MFMAs run, across the
// stage boundary too: the one barrier per k-step sits between the two
// slices of a step, after every wave has read all of that step's
// fragments.
constexpr int BK2 = 32;  // k per stage of the 4-wave kernel = 4 chunks of 8

// k-contiguous rows of 32 elements; chunk c of row r at c ^ ((r >> 2) & 3):
// 16 consecutive rows then cover all 64 banks with one 16-byte read each.
__device__ __forceinline__ int swz4(int row, int chunk) { return chunk ^ ((row >> 2) & 3); }

template <typename T, int R, int NT, bool KC>
struct Dma2;

// k-contiguous: slot q = i*NT + tid of a stage holds row q/4, physical
// chunk q%4.
template <typename T, int R, int NT>
struct Dma2<T, R, NT, true> {
    static constexpr int NV = R * 4 / NT;
    static_assert(NV >= 1 && NV * NT == R * 4, "tile / thread mismatch");
    const T* src[NV];
    int cofs[NV];

    __device__ __forceinline__ void init(const Operand& op, int o0, int omax, int64_t boff) {
        const int tid = threadIdx.x;
#pragma unroll
        for (int i = 0; i < NV; ++i) {
            const int q = i * NT + tid, r = q >> 2, c = swz4(r, q & 3);
            const int o = o0 + r < omax ? o0 + r : (omax > 0 ? omax - 1 : 0);
            int seg = 0;
            const int64_t off = map_off(op.row, (uint32_t)o, op.nseg, &seg);
            src[i] = reinterpret_cast<const T*>(seg_ptr(op.ptr, seg)) + boff + off;
            cofs[i] = c * 8;
        }
    }
    __device__ __forceinline__ void issue(const Operand&, int k0, int kend, uint32_t stage_lds) const {
        const int w = threadIdx.x >> 6;
#pragma unroll
        for (int i = 0; i < NV; ++i) {
            const int k = k0 + cofs[i];
            const void* p = k < kend ? (const void*)(src[i] + k) : (const void*)g_zero16;
            lds_dma16(p, stage_lds + (uint32_t)(i * NT + w * 64) * 16u);
        }
    }
    // lane l: row ob + l%32, k = kk + 8 (l / 32) .. +7
    __device__ __forceinline__ static u32x4 frag(const T* lds, int ob, int kk, int lane) {
        const int r = ob + (lane & 31);
        const int c = (kk >> 3) + (lane >> 5);
        return *reinterpret_cast<const u32x4*>(lds + r * BK2 + swz4(r, c) * 8);
    }
};

// outer-contiguous: [k][outer] rows of R elements, slot q holds k-row q/CPR,
// physical chunk q%CPR = logical chunk ^ (4 (row & 3)); fragments as in
// Frag32<T, R, false>.
template <typename T, int R, int NT>
struct Dma2<T, R, NT, false> {
    static constexpr int CPR = R / 8;
    static constexpr int NV = BK2 * CPR / NT;
    static_assert(NV >= 1 && NV * NT == BK2 * CPR && CPR >= 16, "tile / thread mismatch");
    int kr[NV];
    int oofs[NV];
    int64_t boff;

    __device__ __forceinline__ void init(const Operand&, int o0, int omax, int64_t b) {
        const int tid = threadIdx.x;
        boff = b;
#pragma unroll
        for (int i = 0; i < NV; ++i) {
            const int q = i * NT + tid;
            kr[i] = q / CPR;
            const int c = (q % CPR) ^ (4 * (kr[i] & 3));
            const int o = o0 + c * 8;
            oofs[i] = o < omax ? o : 0;
        }
    }
    __device__ __forceinline__ void issue(const Operand& op, int k0, int kend, uint32_t stage_lds) const {
        const int w = threadIdx.x >> 6;
#pragma unroll
        for (int i = 0; i < NV; ++i) {
            // k0 < kend here, so k0 is a valid row for lanes past the end
            const int k = k0 + kr[i];
            const bool in = k < kend;
            int seg = 0;
            const int64_t off = map_off(op.row, (uint32_t)(in ? k : k0), op.nseg, &seg);
            const T* src = reinterpret_cast<const T*>(seg_ptr(op.ptr, seg)) + boff + off + oofs[i];
            lds_dma16(in ? (const void*)src : (const void*)g_zero16, stage_lds + (uint32_t)(i * NT + w * 64) * 16u);
        }
    }
    __device__ __forceinline__ static u32x4 frag(const T* lds, int ob, int kk, int lane) {
        return Frag32<T, R, false>::read(lds, ob, kk, lane);
    }
};

template <typename T, int WGM, int WGN, bool AKC, bool BKC>
__global__ __launch_bounds__(64 * WGM * WGN) void gemm_big(GemmArgs g) {
    constexpr int BM = 256, BN = 256, NT = 64 * WGM * WGN;
    constexpr int WM = BM / WGM, WN = BN / WGN, FM = WM / 32, FN = WN / 32, STAGES = 4;
    static_assert(WN % 64 == 0, "wave tile must cover whole 64-column passes");
    constexpr int AS = BM * BK2, BS = BN * BK2;
    constexpr int STAGE = (AS + BS) * (int)sizeof(T);
    constexpr int SMEM = STAGES * STAGE;
    static_assert(WGM * WGN * 32 * (WN + 8) * 4 <= SMEM, "epilogue strips do not fit");
    __shared__ __attribute__((aligned(16))) unsigned char smem[SMEM];
    typedef Dma2<T, BM, NT, AKC> DA;
    typedef Dma2<T, BN, NT, BKC> DB;
    constexpr int NL = DA::NV + DB::NV;  // copies per thread per stage
    typedef typename Mfma32<T>::frag frag;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave / WGN, wn = wave % WGN;
    int tm, tn;
    int by;
    tile_of(g.tiles_m, g.tiles_n, tm, tn, by);
    const int m0 = tm * BM, n0 = tn * BN;
    const int splits = g.splits > 1 ? g.splits : 1;
    const uint32_t z = (uint32_t)by / splits;
    const int sidx = by - (int)z * splits;
    const int kb = splits > 1 ? sidx * g.kper : 0;
    const int ke = splits > 1 ? min(g.K, kb + g.kper) : g.K;
    int dummy = 0;
    DA da;
    DB db;
    da.init(g.a, m0, g.M, map_off(g.a.batch, z, 1, &dummy));
    db.init(g.b, n0, g.N, map_off(g.b.batch, z, 1, &dummy));
    const uint32_t base = lds_addr(smem);

    floatx16 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    const int nk = ke > kb ? (ke - kb + BK2 - 1) / BK2 : 0;
    auto issue = [&](int s) {
        const uint32_t st = base + (uint32_t)((s & 3) * STAGE);
        da.issue(g.a, kb + s * BK2, ke, st);
        db.issue(g.b, kb + s * BK2, ke, st + (uint32_t)(AS * sizeof(T)));
    };
    auto stage_a = [&](int s) { return reinterpret_cast<const T*>(smem + (s & 3) * STAGE); };
    frag a0[FM], b0[FN], a1[FM], b1[FN];
    auto read = [&](frag (&a)[FM], frag (&b)[FN], int s, int kk) {
        const T* A = stage_a(s);
        const T* B = A + AS;
#pragma unroll
        for (int i = 0; i < FM; ++i) a[i] = __builtin_bit_cast(frag, DA::frag(A, wm * WM + i * 32, kk, lane));
#pragma unroll
        for (int j = 0; j < FN; ++j) b[j] = __builtin_bit_cast(frag, DB::frag(B, wn * WN + j * 32, kk, lane));
    };
    auto mma = [&](const frag (&a)[FM], const frag (&b)[FN]) {
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
            for (int j = 0; j < FN; ++j) acc[i][j] = Mfma32<T>::run(a[i], b[j], acc[i][j]);
    };

    if (nk > 0) {
        issue(0);
        if (nk > 1) issue(1);
        if (nk > 2) issue(2);
        if (nk > 2) wait_vm<2 * NL>();
        else if (nk > 1) wait_vm<NL>();
        else wait_vm<0>();
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
        read(a0, b0, 0, 0);
    }
    // The fences keep each fragment read ahead of the MFMAs it overlaps (the
    // compiler would otherwise sink the reads to their first use).
    for (int s = 0; s < nk; ++s) {
        // slice 0 of step s; fragments of slice 1 meanwhile
        read(a1, b1, s, 16);
        asm volatile("" ::: "memory");
        __builtin_amdgcn_sched_barrier(0);
        mma(a0, b0);
        // step s+1 must have landed (copies of s+2 may still fly), and this
        // wave's reads of step s are complete before any wave refills a slot
        if (s + 2 < nk) wait_vm<NL>();
        else wait_vm<0>();
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
        if (s + 3 < nk) issue(s + 3);
        // slice 1 of step s; fragments of slice 0 of step s+1 meanwhile
        // (after the last step this reads a stale slot, unused; keeping the
        // read unconditional keeps the LDS wait counts exact)
        read(a0, b0, s + 1, 0);
        asm volatile("" ::: "memory");
        __builtin_amdgcn_sched_barrier(0);
        mma(a1, b1);
        __builtin_amdgcn_sched_barrier(0);
    }
    epilogue_direct<T, WM, WN>(g, acc, m0 + wm * WM, n0 + wn * WN, z, sidx, splits);
}

// ------------------------------------------------------ lean kernels
// 32x32x16-MFMA contractions with BM x BN block tiles, WGM x WGN waves,
// k-steps of BKS (32 or 64) and a ring of STAGES LDS stages filled by
// asynchronous global -> LDS copies STAGES - 1 steps ahead.  Compared with
// the general kernels above, operand addresses are set up so that the
// k-loop does one pointer offset per copy and no bounds test: a
// k-contiguous operand keeps one pointer per row (any row map, evaluated
// once), an outer-contiguous operand's row map must be affine over each
// k-step (one wave-uniform map evaluation per step plus fixed per-thread
// offsets), k must be a multiple of BKS, and rows / columns past M / N
// read a clamped valid row whose results are never stored.  The epilogue
// writes straight from the accumulators with one address per 32x32 block,
// which needs output maps affine over aligned 32-blocks (g.blk32).
// Several waves per SIMD matter here: one wave alone cannot issue LDS
// fragment reads fast enough to keep its MFMAs busy.

// LDS chunk (16 bytes) position of logical chunk c of k-contiguous row r,
// rows of CPR chunks: 16 consecutive rows read at one chunk cover all 64
// banks once.
template <int CPR>
__device__ __forceinline__ int lswz(int r, int c) {
    if constexpr (CPR == 4) return c ^ ((r >> 2) & 3);
    else return c ^ ((r >> 1) & 7);
}

// k-contiguous operand of R rows: slot q = i*NT + tid of a stage holds
// row q / CPR, physical chunk q % CPR.  NT (a power of two) is the number
// of threads that copy the operand: the block's, or the first or second
// half of it (tid = thread index modulo NT).
template <typename T, int R, int BKS, int NT>
struct LeanK {
    static constexpr int CPR = BKS / 8;
    static constexpr int NV = R * CPR / NT;
    static_assert((NT & (NT - 1)) == 0, "copying threads: a power of two");
    static_assert(NV >= 1 && NV * NT == R * CPR, "tile / thread mismatch");
    const T* src[NV];
    __device__ __forceinline__ void init(const Operand& op, int64_t boff, int kb, int o0, int omax) {
        const int tid = threadIdx.x & (NT - 1);
#pragma unroll
        for (int i = 0; i < NV; ++i) {
            const int q = i * NT + tid, r = q / CPR, c = lswz<CPR>(r, q % CPR);
            const int o = o0 + r < omax ? o0 + r : omax - 1;
            int seg = 0;
            const int64_t off = map_off(op.row, (uint32_t)o, op.nseg, &seg);
            src[i] = reinterpret_cast<const T*>(seg_ptr(op.ptr, seg)) + boff + off + kb + c * 8;
        }
    }
    __device__ __forceinline__ void issue(const Operand&, int64_t, int kb, int s, uint32_t st) const {
        const int w = (threadIdx.x & (NT - 1)) >> 6;
#pragma unroll
        for (int i = 0; i < NV; ++i) lds_dma16(src[i] + s * BKS, st + (uint32_t)(i * NT + w * 64) * 16u);
        (void)kb;
    }
    // the same copies one at a time (prep once per step, then copy i)
    __device__ __forceinline__ const T* prep(const Operand&, int64_t, int, int) const { return nullptr; }
    __device__ __forceinline__ void copy(const T*, int s, int i, uint32_t st) const {
        lds_dma16(src[i] + s * BKS, st + (uint32_t)(i * NT + ((threadIdx.x & (NT - 1)) >> 6) * 64) * 16u);
    }
    // lane l: row ob + l % 32, k = kk + 8 (l / 32) .. +7
    __device__ __forceinline__ static u32x4 frag(const T* lds, int ob, int kk, int lane) {
        const int r = ob + (lane & 31);
        const int c = (kk >> 3) + (lane >> 5);
        return *reinterpret_cast<const u32x4*>(lds + r * BKS + lswz<CPR>(r, c) * 8);
    }
};

// outer-contiguous operand ([k][outer] rows of R elements in LDS): slot q
// holds k-row q / CPR, physical chunk q % CPR = logical chunk ^ 4 (row & 3).
template <typename T, int R, int BKS, int NT>
struct LeanO {
    static constexpr int CPR = R / 8;
    static constexpr int NV = BKS * CPR / NT;
    static_assert((NT & (NT - 1)) == 0, "copying threads: a power of two");
    static_assert(NV >= 1 && NV * NT == BKS * CPR, "tile / thread mismatch");
    int64_t poff[NV];  // k-row * stride + outer offset
    __device__ __forceinline__ void init(const Operand& op, int64_t, int, int o0, int omax) {
        const int tid = threadIdx.x & (NT - 1);
#pragma unroll
        for (int i = 0; i < NV; ++i) {
            const int q = i * NT + tid, kr = q / CPR, c = (q % CPR) ^ (4 * (kr & 3));
            const int o = o0 + c * 8 < omax ? o0 + c * 8 : 0;
            poff[i] = (int64_t)kr * op.row.s0 + o;
        }
    }
    __device__ __forceinline__ void issue(const Operand& op, int64_t boff, int kb, int s, uint32_t st) const {
        const int w = (threadIdx.x & (NT - 1)) >> 6;
        int seg = 0;
        const int64_t off = map_off(op.row, (uint32_t)(kb + s * BKS), op.nseg, &seg);
        const T* base = reinterpret_cast<const T*>(seg_ptr(op.ptr, seg)) + boff + off;
#pragma unroll
        for (int i = 0; i < NV; ++i) lds_dma16(base + poff[i], st + (uint32_t)(i * NT + w * 64) * 16u);
    }
    __device__ __forceinline__ const T* prep(const Operand& op, int64_t boff, int kb, int s) const {
        int seg = 0;
        const int64_t off = map_off(op.row, (uint32_t)(kb + s * BKS), op.nseg, &seg);
        return reinterpret_cast<const T*>(seg_ptr(op.ptr, seg)) + boff + off;
    }
    __device__ __forceinline__ void copy(const T* base, int, int i, uint32_t st) const {
        lds_dma16(base + poff[i], st + (uint32_t)(i * NT + ((threadIdx.x & (NT - 1)) >> 6) * 64) * 16u);
    }
    __device__ __forceinline__ static u32x4 frag(const T* lds, int ob, int kk, int lane) {
        return Frag32<T, R, false>::read(lds, ob, kk, lane);
    }
};

template <typename T, int R, int BKS, int NT, bool KC>
struct LeanSel { typedef LeanK<T, R, BKS, NT> type; };
template <typename T, int R, int BKS, int NT>
struct LeanSel<T, R, BKS, NT, false> { typedef LeanO<T, R, BKS, NT> type; };

// Output addressing of the lean epilogue (also used for split-k partials:
// row-major floats, one pointer).
struct LeanOut {
    void* ptr[3];
    int nseg, seg_on_m, affine, cn;
    int64_t ldc, coff;
    IdxMap mmap, nmap;
};

// Stores of one wave's tile straight from the accumulators (a 32x32 result
// holds column l % 32 in lane l at rows 8 (r / 4) + 4 (l / 32) + r % 4):
// along n, the 32 lanes of a half-wave write 32 consecutive elements of a
// row; along m, each lane writes the 4 consecutive rows of a group as one
// vector.  One address per 32x32 block (row part wave-uniform).  M is a
// multiple of 8, so a group of 4 rows is wholly inside or outside.
template <typename OutT, bool CN, int FM, int FN>
__device__ __forceinline__ void lean_store(const GemmArgs& g, const LeanOut& o, const floatx16 (&acc)[FM][FN],
                                           int mw, int nw, const float (&bn)[FN], float alpha,
                                           const floatx16 (*res)[FN] = nullptr) {
    const int lane = threadIdx.x & 63, c = lane & 31, h = lane >> 5;
    const int64_t rs = o.affine ? (CN ? o.ldc : 1) : o.mmap.s0;
#pragma unroll
    for (int i = 0; i < FM; ++i) {
        const int mb = mw + i * 32;
        if (mb >= g.M) break;
        int mseg = 0;
        const int64_t rbase = o.affine ? (int64_t)mb * rs : map_off(o.mmap, (uint32_t)mb, o.seg_on_m ? o.nseg : 1, &mseg);
#pragma unroll
        for (int j = 0; j < FN; ++j) {
            const int n = nw + j * 32 + c;
            if (n >= g.N) continue;
            int nsg = 0;
            const int64_t ncol = o.affine ? (CN ? (int64_t)n : (int64_t)n * o.ldc)
                                          : map_off(o.nmap, (uint32_t)n, o.seg_on_m ? 1 : o.nseg, &nsg);
            OutT* pb = reinterpret_cast<OutT*>(seg_ptr(o.ptr, o.seg_on_m ? mseg : nsg)) + o.coff + rbase + ncol +
                       (CN ? (int64_t)(4 * h) * rs : (int64_t)(4 * h));
#pragma unroll
            for (int rg = 0; rg < 4; ++rg) {
                if (mb + 8 * rg + 4 * h >= g.M) continue;
                float v[4];
#pragma unroll
                for (int k = 0; k < 4; ++k) v[k] = acc[i][j][4 * rg + k] * alpha + bn[j] + (res ? res[i][j][4 * rg + k] : 0.f);
                if constexpr (CN) {
#pragma unroll
                    for (int k = 0; k < 4; ++k) pb[(int64_t)(8 * rg + k) * rs] = from_f<OutT>(v[k]);
                } else if constexpr (sizeof(OutT) == 4) {
                    floatx4 ov = {v[0], v[1], v[2], v[3]};
                    *reinterpret_cast<floatx4*>(pb + 8 * rg) = ov;
                } else {
                    OutT o4[4];
#pragma unroll
                    for (int k = 0; k < 4; ++k) o4[k] = from_f<OutT>(v[k]);
                    *reinterpret_cast<u32x2*>(pb + 8 * rg) = __builtin_bit_cast(u32x2, o4);
                }
            }
        }
    }
}

// Stores through LDS (row-major output, one pointer, N and the row pitch
// multiples of 8): each 32-row block of the wave's tile is written to the
// wave's own LDS region in its accumulator layout (rows padded by 32 bytes,
// so the two half-waves' rows fall on disjoint banks), then read back as
// 16-byte row pieces, so every global store instruction writes whole
// 128-byte lines.  A wave's LDS accesses run in order, so no barrier is
// needed between its writes and reads.
// ACT (Epilogue::act_mode) 1: also the activation output of each stored
// piece; 2: the activation backward of each piece stored in its place,
// with the lane's column sums over its rows added across the wave's lanes
// at the end (partial row mw / (FM * 32)).  The read-back loop of these
// is not unrolled, so the accumulator loop stays small enough to unroll
// (the accumulators must stay in registers).
template <typename OutT, int FM, int FN, int ACT = 0>
__device__ __forceinline__ void lean_store_staged(const GemmArgs& g, const LeanOut& o, const floatx16 (&acc)[FM][FN],
                                                  int mw, int nw, const float (&bn)[FN], float alpha,
                                                  unsigned char* region) {
    constexpr int WN = FN * 32, LDR = WN + 32 / (int)sizeof(OutT);  // row pitch in elements
    // rows per read pass (lanes past RPI * VPR idle when VPR does not divide 64)
    constexpr int EPV = 16 / (int)sizeof(OutT), VPR = WN / EPV, RPI = 64 / VPR, NPASS = (32 + RPI - 1) / RPI;
    static_assert(VPR <= 64 && WN % EPV == 0, "staged store shape");
    OutT* sm = reinterpret_cast<OutT*>(region);
    const int lane = threadIdx.x & 63, c = lane & 31, h = lane >> 5;
    const int rr0 = lane / VPR, vc = (lane % VPR) * EPV;
    OutT* out = reinterpret_cast<OutT*>(o.ptr[0]) + o.coff;
    // (an output through index maps: the column part of a piece's address
    // is the lane's for the whole tile, the row part is taken per row)
    int nseg = 0;
    int64_t noff = 0;
    if (!o.affine && nw + vc < g.N)
        noff = map_off(o.nmap, (uint32_t)(nw + vc), o.seg_on_m ? 1 : o.nseg, &nseg);
    auto piece = [&](int m) -> OutT* {
        if (o.affine) return out + (int64_t)m * o.ldc + nw + vc;
        int mseg = 0;
        const int64_t moff = map_off(o.mmap, (uint32_t)m, o.seg_on_m ? o.nseg : 1, &mseg);
        return reinterpret_cast<OutT*>(seg_ptr(o.ptr, o.seg_on_m ? mseg : nseg)) + o.coff + moff + noff;
    };
    float cs[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) cs[q] = 0.f;
    // activation step: the bias of the lane's 8 columns is the same for
    // every row of the tile (loaded once, kept packed)
    const bool lane_on = lane < RPI * VPR && nw + vc < g.N;
    u32x4 bias_raw = {0u, 0u, 0u, 0u};
    if constexpr (ACT != 0)
        if (lane_on) bias_raw = *reinterpret_cast<const u32x4*>(reinterpret_cast<const OutT*>(g.c.act_bias) + nw + vc);

#pragma unroll
    for (int i = 0; i < FM; ++i) {
        const int mb = mw + i * 32;
        if (mb >= g.M) break;
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int rr = 8 * (r >> 2) + 4 * h + (r & 3);
                sm[rr * LDR + j * 32 + c] = from_f<OutT>(acc[i][j][r] * alpha + bn[j]);
            }
        // mode 2: the block's pre-activation pieces, all requested before
        // the first is used (once the block's accumulators are in LDS, so
        // that they do not add to the registers held)
        u32x4 hv[ACT == 2 ? NPASS : 1];
        if constexpr (ACT == 2) {
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int p = 0; p < NPASS; ++p) {
                const int rr = p * RPI + rr0;
                hv[p] = u32x4{0u, 0u, 0u, 0u};
                if (lane_on && rr < 32 && mb + rr < g.M)
                    hv[p] = *reinterpret_cast<const u32x4*>(reinterpret_cast<const OutT*>(g.c.act_in) + o.coff +
                                                            (int64_t)(mb + rr) * o.ldc + nw + vc);
            }
        }
        const int n = nw + vc;
        if constexpr (ACT == 0) {
#pragma unroll
            for (int p = 0; p < NPASS; ++p) {
                const int rr = p * RPI + rr0;
                if (lane < RPI * VPR && rr < 32) {
                    const u32x4 v = *reinterpret_cast<const u32x4*>(sm + rr * LDR + vc);
                    if (mb + rr < g.M && n < g.N) *reinterpret_cast<u32x4*>(piece(mb + rr)) = v;
                }
            }
        } else {
            static_assert(sizeof(OutT) == 2, "activation step in a 16-bit type");
            // (passes not unrolled, so that the accumulators of the blocks
            // still to store stay in registers: the pass's pre-activation
            // piece is taken from the front of hv, which then shifts)
#pragma unroll 1
            for (int p = 0; p < NPASS; ++p) {
                const int rr = p * RPI + rr0;
                const u32x4 hcur = hv[0];
#pragma unroll
                for (int t = 0; t + 1 < (ACT == 2 ? NPASS : 1); ++t) hv[t] = hv[t + 1];
                if (lane < RPI * VPR && rr < 32) {
                    const u32x4 v = *reinterpret_cast<const u32x4*>(sm + rr * LDR + vc);
                    if (mb + rr < g.M && n < g.N) {
                        const int64_t off = (int64_t)(mb + rr) * o.ldc + n;
                        float a[8], b[8];
                        V8<OutT>::unpack(v, a);
                        V8<OutT>::unpack(bias_raw, b);
                        if constexpr (ACT == 1) {
                            // the stored values, then their activation (the bias +
                            // activation operator's arithmetic, element index
                            // off .. off+7)
                            *reinterpret_cast<u32x4*>(out + off) = v;
#pragma unroll
                            for (int q = 0; q < 8; ++q) a[q] = act_fwd(a[q] + b[q], g.c.act);
                            dropout8(g.c.act_dp, (uint64_t)off, a);
                            V8<OutT>::store(reinterpret_cast<OutT*>(g.c.act_out) + o.coff + off, a);
                        } else {
                            // the activation backward of the (rounded) dA: the
                            // activation backward operator's arithmetic
                            float u[8];
                            V8<OutT>::unpack(hcur, u);
                            dropout8(g.c.act_dp, (uint64_t)off, a);
#pragma unroll
                            for (int q = 0; q < 8; ++q) {
                                a[q] = to_f(from_f<OutT>(a[q] * act_grad(u[q] + b[q], g.c.act)));
                                cs[q] += a[q];
                            }
                            V8<OutT>::store(out + off, a);
                        }
                    }
                }
            }
        }
    }
    if constexpr (ACT == 2) {
        // lanes with the same 8 columns differ by multiples of VPR
        static_assert((VPR & (VPR - 1)) == 0, "column groups of a power-of-two lane count");
#pragma unroll
        for (int d = VPR; d < 64; d <<= 1)
#pragma unroll
            for (int q = 0; q < 8; ++q) cs[q] += __shfl_xor(cs[q], d, 64);
        const int n = nw + vc;
        if (lane < VPR && n < g.N)
            V8<float>::store(g.c.act_part + (int64_t)(mw / (FM * 32)) * g.N + n, cs);
    }
}

// Epilogue of a lean kernel for one wave's FM x FN accumulator blocks at
// (mw, nw): split-k partials as row-major floats through the same store
// routine as float outputs (one code path keeps registers few).  region:
// this wave's LDS for the staged stores (nullptr: straight stores).
template <typename T, int FM, int FN, int ACT = 0>
__device__ __forceinline__ void lean_epilogue(const GemmArgs& g, const floatx16 (&acc)[FM][FN], int mw, int nw,
                                              uint32_t z, int sidx, int splits, unsigned char* region = nullptr) {
    const int lane = threadIdx.x & 63, c = lane & 31;
    int dummy = 0;
    const Epilogue& e = g.c;
    const bool part = splits > 1;
    float bn[FN];
#pragma unroll
    for (int j = 0; j < FN; ++j) {
        const int n = nw + j * 32 + c;
        bn[j] = 0.f;
        if (!part && e.bias[0]) {
            int bseg = 0;
            const int64_t bo = map_off(e.bias_map, (uint32_t)(n < g.N ? n : 0), e.bias_nseg, &bseg);
            bn[j] = to_f(reinterpret_cast<const T*>(seg_ptr(e.bias, bseg))[bo]);
        }
    }
    LeanOut o;
    if (part) {
        o.ptr[0] = o.ptr[1] = o.ptr[2] = g.split_ws + ((int64_t)sidx * g.batch + z) * g.M * (int64_t)g.N;
        o.nseg = 1; o.seg_on_m = 0; o.affine = 1; o.cn = 1; o.ldc = g.N; o.coff = 0;
        o.mmap = e.mmap; o.nmap = e.nmap;
    } else {
        o.ptr[0] = e.ptr[0]; o.ptr[1] = e.ptr[1]; o.ptr[2] = e.ptr[2];
        o.nseg = e.nseg; o.seg_on_m = e.seg_on_m; o.affine = g.affine; o.cn = e.contig_n; o.ldc = g.ldc;
        o.coff = map_off(e.batch, z, 1, &dummy);
        o.mmap = e.mmap; o.nmap = e.nmap;
    }
    const float alpha = part ? 1.0f : e.alpha;
    if constexpr (FM * FN <= 4) {
        // residual operand (same addressing as the output, along n, input
        // dtype): every value of the wave's tile is loaded before the first
        // store, since vector-memory waits count loads and stores together
        if (!part && e.resid && o.cn && !e.out_f32) {
            floatx16 res[FM][FN];
            const int h = lane >> 5;
#pragma unroll
            for (int i = 0; i < FM; ++i) {
                const int mb = mw + i * 32;
                int mseg = 0;
                const int64_t rs = o.affine ? o.ldc : o.mmap.s0;
                const int64_t rbase = o.affine ? (int64_t)(mb < g.M ? mb : 0) * rs
                                               : map_off(o.mmap, (uint32_t)(mb < g.M ? mb : 0), 1, &mseg);
#pragma unroll
                for (int j = 0; j < FN; ++j) {
                    const int n = nw + j * 32 + c;
                    int nsg = 0;
                    const int64_t ncol = o.affine ? (int64_t)(n < g.N ? n : 0)
                                                  : map_off(o.nmap, (uint32_t)(n < g.N ? n : 0), 1, &nsg);
                    // unconditional loads (a clamped offset for elements
                    // outside the output, whose values are never stored), so
                    // all of them are in flight before the first wait
                    const T* rp = reinterpret_cast<const T*>(e.resid) + o.coff;
                    const int64_t boff = rbase + ncol;
#pragma unroll
                    for (int r = 0; r < 16; ++r) {
                        const int rr = 8 * (r >> 2) + 4 * h + (r & 3);
                        const bool in = mb + rr < g.M && n < g.N;
                        res[i][j][r] = to_f(rp[in ? boff + (int64_t)rr * rs : 0]);
                    }
                }
            }
            lean_store<T, true, FM, FN>(g, o, acc, mw, nw, bn, alpha, res);
            return;
        }
    }
    if (region) {
        if constexpr (ACT != 0) lean_store_staged<T, FM, FN, ACT>(g, o, acc, mw, nw, bn, alpha, region);
        else if (part || e.out_f32) lean_store_staged<float, FM, FN>(g, o, acc, mw, nw, bn, alpha, region);
        else lean_store_staged<T, FM, FN>(g, o, acc, mw, nw, bn, alpha, region);
        return;
    }
    if (part || (o.cn && e.out_f32)) lean_store<float, true, FM, FN>(g, o, acc, mw, nw, bn, alpha);
    else if (o.cn) lean_store<T, true, FM, FN>(g, o, acc, mw, nw, bn, alpha);
    else if (e.out_f32) lean_store<float, false, FM, FN>(g, o, acc, mw, nw, bn, alpha);
    else lean_store<T, false, FM, FN>(g, o, acc, mw, nw, bn, alpha);
}


// KG > 1 splits each k-step's 16-wide slices among KG groups of WGM x WGN
// waves (group g takes slices g, g + KG, ...), so a wave holds a larger
// tile of the output and reads fewer fragments per MFMA; the groups' fp32
// partial tiles are added through LDS before the stores.
template <typename T, int BM, int BN, int WGM, int WGN, int BKS, int STAGES, bool AKC, bool BKC, int KG,
          bool RS = false, int SCH = 0, int ACT = 0>
__device__ __forceinline__ void lean_run(const GemmArgs& g, int tm, int tn, int by) {
    // k-loop schedule: 0 reads next to MFMAs, 1 interleaved (one wave per
    // SIMD), 2 ping-pong (two wave groups alternating)
    constexpr bool IL = SCH == 1, PP = SCH == 2;
    constexpr int NT = 64 * WGM * WGN * KG, WM = BM / WGM, WN = BN / WGN, FM = WM / 32, FN = WN / 32;
    constexpr int NQ = BKS / 16;  // 16-wide k slices per step
    constexpr int NQL = NQ / KG;  // of them, the slices of one wave
    static_assert(NQL * KG == NQ && NQL % 2 == 0 && (KG == 1 || (KG == 2 && FM % 2 == 0)), "k groups");
    constexpr int AS = BM * BKS, BS = BN * BKS;
    constexpr int STAGE = (AS + BS) * (int)sizeof(T);
    static_assert(STAGES >= 3 && FM >= 1 && FN >= 1 && STAGES * STAGE <= 160 * 1024, "configuration");
    __shared__ __attribute__((aligned(16))) unsigned char smem[STAGES * STAGE];
    // (the ping-pong schedule copies each operand with half of the threads)
    constexpr int NTC = PP ? NT / 2 : NT;
    typedef typename LeanSel<T, BM, BKS, NTC, AKC>::type DA;
    typedef typename LeanSel<T, BN, BKS, NTC, BKC>::type DB;
    constexpr int NL = DA::NV + DB::NV;  // copies per thread per step
    typedef typename Mfma32<T>::frag frag;

    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int kg = wave / (WGM * WGN), wl = wave - kg * (WGM * WGN);
    const int wm = wl / WGN, wn = wl % WGN;
    const int m0 = tm * BM, n0 = tn * BN;
    const int splits = g.splits > 1 ? g.splits : 1;
    const uint32_t z = (uint32_t)by / splits;
    const int sidx = by - (int)z * splits;
    const int kb = splits > 1 ? sidx * g.kper : 0;
    const int ke = splits > 1 ? min(g.K, kb + g.kper) : g.K;
    int dummy = 0;
    const int64_t aoff = map_off(g.a.batch, z, 1, &dummy), boff = map_off(g.b.batch, z, 1, &dummy);
    DA da;
    DB db;
    da.init(g.a, aoff, kb, m0, g.M);
    db.init(g.b, boff, kb, n0, g.N);
    const uint32_t base = lds_addr(smem);

    floatx16 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
    // RS: partial row sums of A over the contraction (Epilogue::rsum).  The
    // waves of one tile row (tiles_n blocks x WGN waves that read the same
    // A rows) share its 16-wide k slices round robin: wave wn of block tn
    // adds up the A fragments of slices u = s * NQL + q with
    // u % (tiles_n * WGN) == tn * WGN + wn (a fragment covers 16 k of 32
    // rows, the two lane halves complementary k) and writes partial row
    // tn * WGN + wn.
    static_assert(!RS || KG == 1, "row sums need a single k group");
    const bool rsum = RS && g.c.rsum != nullptr;
    const int rs_nw = g.tiles_n * WGN;
    int rs_next = tn * WGN + wn;
    float rs[FM];
#pragma unroll
    for (int i = 0; i < FM; ++i) rs[i] = 0.f;

    const int nk = (ke - kb) / BKS;
    auto issue = [&](int s) {
        const uint32_t st = base + (uint32_t)((s % STAGES) * STAGE);
        da.issue(g.a, aoff, kb, s, st);
        db.issue(g.b, boff, kb, s, st + (uint32_t)(AS * sizeof(T)));
    };
    frag a[2][FM], b[2][FN];
    auto read = [&](int buf, int s, int q) {
        const T* A = reinterpret_cast<const T*>(smem + (s % STAGES) * STAGE);
        const T* B = A + AS;
#pragma unroll
        for (int i = 0; i < FM; ++i) a[buf][i] = __builtin_bit_cast(frag, DA::frag(A, wm * WM + i * 32, q * 16, lane));
#pragma unroll
        for (int j = 0; j < FN; ++j) b[buf][j] = __builtin_bit_cast(frag, DB::frag(B, wn * WN + j * 32, q * 16, lane));
    };
    auto mma = [&](int buf) {
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
            for (int j = 0; j < FN; ++j) acc[i][j] = Mfma32<T>::run(a[buf][i], b[buf][j], acc[i][j]);
    };

    if (!PP && nk > 0) {
#pragma unroll
        for (int s = 0; s < STAGES - 1; ++s)
            if (s < nk) issue(s);
        if (nk >= STAGES - 1) wait_vm<(STAGES - 2) * NL>();
        else wait_vm<0>();
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
        read(0, 0, kg);
    }
    // IL (one wave per SIMD): every MFMA of a slice is issued next to its
    // share of the next slice's fragment reads (and, in the last slice of
    // a step, of the next step's copies), so the wave keeps its MFMA unit
    // busy while LDS and memory work proceed.  Half of the last slice's
    // MFMAs go before the step barrier.  No LDS wait is needed at the
    // barrier: the slot refilled is that of step s-1, whose reads every
    // wave has consumed (its MFMAs were issued) before reaching it.
    static_assert(!IL || (KG == 1 && !RS), "interleaved schedule: single k group, no row sums");
    if constexpr (IL) {
        constexpr int NMF = FM * FN, NR = FM + FN, H = NMF / 2, R2 = NMF - H;
        // fragment reads / copies per MFMA (fixed trip counts, so every
        // loop unrolls and every register array index is a constant)
        constexpr int RPM = (NR + NMF - 1) / NMF, RPL = (NR + R2 - 1) / R2, CPL = (NL + R2 - 1) / R2;
        // read j of a slice, in the order the slice's MFMAs (t -> a[t / FN],
        // b[t % FN]) first need them: a0, b0 .. b(FN-1), a1 .. a(FM-1)
        auto read_one = [&](int buf, int s, int q, int j) {
            const T* A = reinterpret_cast<const T*>(smem + (s % STAGES) * STAGE);
            const T* B = A + AS;
            if (j >= 1 && j <= FN)
                b[buf][j - 1] = __builtin_bit_cast(frag, DB::frag(B, wn * WN + (j - 1) * 32, q * 16, lane));
            else {
                const int i = j == 0 ? 0 : j - FN;
                a[buf][i] = __builtin_bit_cast(frag, DA::frag(A, wm * WM + i * 32, q * 16, lane));
            }
        };
        auto mma_one = [&](int buf, int t) {
            acc[t / FN][t % FN] = Mfma32<T>::run(a[buf][t / FN], b[buf][t % FN], acc[t / FN][t % FN]);
        };
        for (int s = 0; s < nk; ++s) {
#pragma unroll
            for (int q = 0; q < NQL; ++q) {
                const int cur = q & 1;
                if (q + 1 < NQL) {
#pragma unroll
                    for (int t = 0; t < NMF; ++t) {
                        mma_one(cur, t);
#pragma unroll
                        for (int jj = 0; jj < RPM; ++jj)
                            if (t * RPM + jj < NR) read_one(cur ^ 1, s, q + 1, t * RPM + jj);
                        __builtin_amdgcn_sched_barrier(0);
                    }
                } else {
#pragma unroll
                    for (int t = 0; t < H; ++t) mma_one(cur, t);
                    __builtin_amdgcn_sched_barrier(0);
                    if (s + STAGES - 2 < nk) wait_vm<(STAGES - 3) * NL>();
                    else wait_vm<0>();
                    __builtin_amdgcn_s_barrier();
                    asm volatile("" ::: "memory");
                    __builtin_amdgcn_sched_barrier(0);
                    const int sn = s + STAGES - 1;
                    const bool more = sn < nk;
                    const uint32_t st = base + (uint32_t)((sn % STAGES) * STAGE);
                    const T* pa = da.prep(g.a, aoff, kb, sn);
                    const T* pb = db.prep(g.b, boff, kb, sn);
#pragma unroll
                    for (int u = 0; u < R2; ++u) {
                        mma_one(cur, H + u);
                        if (more) {
#pragma unroll
                            for (int cc = 0; cc < CPL; ++cc) {
                                const int c = u * CPL + cc;
                                if (c < DA::NV) da.copy(pa, sn, c, st);
                                else if (c < NL) db.copy(pb, sn, c - DA::NV, st + (uint32_t)(AS * sizeof(T)));
                            }
                        }
#pragma unroll
                        for (int jj = 0; jj < RPL; ++jj)
                            if (u * RPL + jj < NR) read_one(cur ^ 1, s + 1, 0, u * RPL + jj);
                        __builtin_amdgcn_sched_barrier(0);
                    }
                }
            }
        }
    } else if constexpr (PP) {
        // PP (two waves per SIMD): the waves of the upper half of the tile
        // (group 0, one per SIMD) and of the lower half (group 1) alternate
        // between a memory phase
        // (every fragment of a k-step read from LDS into registers, plus the
        // group's copies of a later step: group 0 copies the A part of every
        // stage, group 1 the B part) and an MFMA phase (the k-step's MFMAs
        // from registers), group 1 one phase behind, so that on each SIMD one
        // wave reads while the other multiplies.  Every phase ends at a block
        // barrier.  Stage s is read in phases 2s (group 0) and 2s+1 (group 1)
        // and its reads complete within the reading group's next (MFMA)
        // phase; its slot is refilled with step s + STAGES from phase 2s + 4
        // on (copies run STAGES - 2 steps ahead).  A group's copies of step
        // s + 1 have landed when its memory phase of step s ends (before that
        // phase's barrier).
        static_assert(KG == 1 && !RS && WGM * WGN == 8 && WGM % 2 == 0,
                      "ping-pong schedule: 8 waves in an even number of wave rows, single k group");
        static_assert(STAGES >= 3, "ping-pong schedule: a stage read, one in flight, one being refilled");
        constexpr int D = STAGES - 2, NH = NT / 2;
        typedef typename LeanSel<T, BM, BKS, NH, AKC>::type PA;
        typedef typename LeanSel<T, BN, BKS, NH, BKC>::type PB;
        // waves 0-3 (the upper half of the wave rows) and 4-7 land on the
        // four SIMDs in the same order: one wave of each group per SIMD
        const int grp = wm / (WGM / 2);
        PA pa;
        PB pb;
        if (grp == 0) pa.init(g.a, aoff, kb, m0, g.M);
        else pb.init(g.b, boff, kb, n0, g.N);
        auto issue_part = [&](int s) {
            const uint32_t st = base + (uint32_t)((s % STAGES) * STAGE);
            if (grp == 0) pa.issue(g.a, aoff, kb, s, st);
            else pb.issue(g.b, boff, kb, s, st + (uint32_t)(AS * sizeof(T)));
        };
        // the group's copies of the oldest step in flight have landed
        auto wait_part = [&](bool more) {
            if (!more) wait_vm<0>();
            else if (grp == 0) wait_vm<(D - 1) * PA::NV>();
            else wait_vm<(D - 1) * PB::NV>();
        };
        frag fa[NQ][FM], fb[NQ][FN];
#pragma unroll
        for (int s = 0; s < D; ++s)
            if (s < nk) issue_part(s);
        wait_part(nk >= D);
        __builtin_amdgcn_s_barrier();
        if (grp == 1 && nk > 0) __builtin_amdgcn_s_barrier();  // group 1 sits out the first phase
        asm volatile("" ::: "memory");
        for (int s = 0; s < nk; ++s) {
            __builtin_amdgcn_sched_barrier(0);
            const T* A = reinterpret_cast<const T*>(smem + (s % STAGES) * STAGE);
            const T* B = A + AS;
#pragma unroll
            for (int q = 0; q < NQ; ++q) {
#pragma unroll
                for (int i = 0; i < FM; ++i) fa[q][i] = __builtin_bit_cast(frag, DA::frag(A, wm * WM + i * 32, q * 16, lane));
#pragma unroll
                for (int j = 0; j < FN; ++j) fb[q][j] = __builtin_bit_cast(frag, DB::frag(B, wn * WN + j * 32, q * 16, lane));
            }
            const bool more = s + D < nk;
            if (more) issue_part(s + D);
            wait_part(more);
            // (the last step's reads complete before the barrier: past it
            // the other group's waves may stage their outputs in LDS)
            if (s + 1 == nk) asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
            __builtin_amdgcn_s_barrier();
            asm volatile("" ::: "memory");
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int q = 0; q < NQ; ++q)
#pragma unroll
                for (int i = 0; i < FM; ++i)
#pragma unroll
                    for (int j = 0; j < FN; ++j) acc[i][j] = Mfma32<T>::run(fa[q][i], fb[q][j], acc[i][j]);
            __builtin_amdgcn_sched_barrier(0);
            // (group 1's last MFMA phase has no partner phase to end)
            if (grp == 0 || s + 1 < nk) __builtin_amdgcn_s_barrier();
            asm volatile("" ::: "memory");
        }
    } else
    // Every 16-wide slice: the next slice's fragments are read while this
    // slice's MFMAs run.  Before the last slice of step s, once step s+1 has
    // landed and this wave's reads of step s are done, one barrier lets the
    // slot of step s-1 be refilled with step s+STAGES-1 (after the last step
    // the read is of a stale slot, unused).
    for (int s = 0; s < nk; ++s) {
#pragma unroll
        for (int q = 0; q < NQL; ++q) {
            const int cur = q & 1;
            if (q + 1 < NQL) {
                read(cur ^ 1, s, (q + 1) * KG + kg);
            } else {
                if (s + STAGES - 2 < nk) wait_vm<(STAGES - 3) * NL>();
                else wait_vm<0>();
                asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
                __builtin_amdgcn_s_barrier();
                asm volatile("" ::: "memory");
                if (s + STAGES - 1 < nk) issue(s + STAGES - 1);
                read(cur ^ 1, s + 1, kg);
            }
            asm volatile("" ::: "memory");
            __builtin_amdgcn_sched_barrier(0);
            mma(cur);
            __builtin_amdgcn_sched_barrier(0);
            if constexpr (RS) {
                if (rsum && s * NQL + q == rs_next) {
#pragma unroll
                    for (int i = 0; i < FM; ++i)
#pragma unroll
                        for (int t = 0; t < 8; ++t) rs[i] += (float)a[cur][i][t];
                    rs_next += rs_nw;
                }
            }
        }
    }

    const int mw = m0 + wm * WM, nw = n0 + wn * WN;
    if constexpr (KG == 1) {
        if (RS && rsum) {
            float* prow = g.c.rsum + (int64_t)(tn * WGN + wn) * g.c.rsum_ld;
#pragma unroll
            for (int i = 0; i < FM; ++i) {
                const float v = rs[i] + __shfl_xor(rs[i], 32, 64);
                const int m = mw + i * 32 + lane;
                if (lane < 32 && m < g.M) prow[m] = v;
            }
        }
        // staged stores: every wave is done with the stages (its reads
        // consumed, the last ones of a stale slot completed) before any
        // wave reuses their LDS; each wave then owns 32 rows of its tile
        // width (padded) at a time
        unsigned char* region = nullptr;
        if (g.ep_stage & (splits > 1 ? 2 : 5)) {
            constexpr int OB = WN * 4 + 32;  // bytes per staged row, float output
            static_assert(32 * OB * WGM * WGN <= STAGES * STAGE, "staging region");
            // (after the ping-pong loop every LDS read and copy completed
            // before the last barrier both groups passed)
            if constexpr (!PP) {
                asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
                __builtin_amdgcn_s_barrier();
                asm volatile("" ::: "memory");
            }
            region = smem + wl * 32 * OB;
        }
        lean_epilogue<T, FM, FN, ACT>(g, acc, mw, nw, z, sidx, splits, region);
    } else {
        // group 0 stores rows [0, FM/2) of the wave tile and group 1 the
        // rest: each group first hands the other half of its partial tile
        // to its partner wave through LDS (the stages are free once every
        // wave has passed the barrier)
        constexpr int FH = FM / 2, SLOT = FH * FN * 16 * 64;
        float* red = reinterpret_cast<float*>(smem);
        auto put = [&](float* dst, auto give_c) {
            constexpr int give = decltype(give_c)::value;
#pragma unroll
            for (int i = 0; i < FH; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j)
#pragma unroll
                    for (int r4 = 0; r4 < 4; ++r4) {
                        floatx4 v = {acc[give + i][j][4 * r4], acc[give + i][j][4 * r4 + 1], acc[give + i][j][4 * r4 + 2],
                                     acc[give + i][j][4 * r4 + 3]};
                        *reinterpret_cast<floatx4*>(dst + (((i * FN + j) * 4 + r4) * 64 + lane) * 4) = v;
                    }
        };
        floatx16 half[FH][FN];
        auto take = [&](const float* src, auto keep_c) {
            constexpr int keep = decltype(keep_c)::value;
#pragma unroll
            for (int i = 0; i < FH; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j)
#pragma unroll
                    for (int r4 = 0; r4 < 4; ++r4) {
                        const floatx4 v = *reinterpret_cast<const floatx4*>(src + (((i * FN + j) * 4 + r4) * 64 + lane) * 4);
#pragma unroll
                        for (int t = 0; t < 4; ++t) half[i][j][4 * r4 + t] = acc[keep + i][j][4 * r4 + t] + v[t];
                    }
        };
        __syncthreads();
        float* to_partner = red + ((1 - kg) * (WGM * WGN) + wl) * SLOT;
        if (kg == 0) put(to_partner, std::integral_constant<int, FH>{});
        else put(to_partner, std::integral_constant<int, 0>{});
        __syncthreads();
        const float* mine = red + (kg * (WGM * WGN) + wl) * SLOT;
        if (kg == 0) take(mine, std::integral_constant<int, 0>{});
        else take(mine, std::integral_constant<int, FH>{});
        lean_epilogue<T, FH, FN>(g, half, mw + kg * FH * 32, nw, z, sidx, splits);
    }
}

template <typename T, int BM, int BN, int WGM, int WGN, int BKS, int STAGES, bool AKC, bool BKC, int KG,
          bool RS = false, int SCH = 0, int ACT = 0>
__global__ __launch_bounds__(64 * WGM * WGN * KG) void gemm_lean(GemmArgs g) {
    int tm, tn, by;
    tile_of(g.tiles_m, g.tiles_n, tm, tn, by);
    lean_run<T, BM, BN, WGM, WGN, BKS, STAGES, AKC, BKC, KG, RS, SCH, ACT>(g, tm, tn, by);
}

// Two unbatched, unsplit contractions in one launch: blocks (renumbered
// over the 8 XCDs as a whole) below g0's tile count take g0's tiles, the
// rest g1's, so two contractions that each leave CUs idle fill the chip
// together.
template <typename T, int BM, int BN, int WGM, int WGN, int BKS, int STAGES, bool AKC, bool BKC, bool RS = false>
__global__ __launch_bounds__(64 * WGM * WGN) void gemm_lean_pair(GemmArgs g0, GemmArgs g1) {
    const int n0 = g0.tiles_m * g0.tiles_n, total = n0 + g1.tiles_m * g1.tiles_n;
    const int lid = xcd_order((int)blockIdx.x, total);
    int tm, tn;
    if (lid < n0) {
        tile_in(lid, g0.tiles_m, g0.tiles_n, tm, tn);
        lean_run<T, BM, BN, WGM, WGN, BKS, STAGES, AKC, BKC, 1, RS>(g0, tm, tn, 0);
    } else {
        tile_in(lid - n0, g1.tiles_m, g1.tiles_n, tm, tn);
        // (same instance as g0's, so that both share one LDS allocation)
        lean_run<T, BM, BN, WGM, WGN, BKS, STAGES, AKC, BKC, 1, RS>(g1, tm, tn, 0);
    }
}

// True when a lean kernel with k-steps of bks takes this contraction.
bool lean_ok(const GemmArgs& g, int bks) {
    const Epilogue& e = g.c;
    if (g.K % bks || (g.splits > 1 && g.kper % bks)) return false;
    // outer-contiguous operands: row map affine over every k-step
    if (!g.a.kcontig && g.a.row.r0 % bks) return false;
    if (!g.b.kcontig && g.b.row.r0 % bks) return false;
    if (!g.blk32 || (e.bias[0] && e.bias_on_m)) return false;
    // a residual operand: only on the 128x128 tile (small wave tiles), along
    // n, in the input dtype, through a single pointer
    if (e.resid && (bks != 64 || !e.contig_n || e.out_f32 || e.nseg != 1)) return false;
    return true;
}

// Sum of the split-K partials in split order, then the regular epilogue.
template <typename T>
__global__ __launch_bounds__(256) void splitk_reduce(GemmArgs g) {
    const int64_t MN8 = (int64_t)g.M * g.N / 8;
    const int64_t total = MN8 * g.batch;
    const int64_t plane = (int64_t)g.batch * g.M * g.N;
    for (int64_t v = (int64_t)blockIdx.x * 256 + threadIdx.x; v < total; v += (int64_t)gridDim.x * 256) {
        const int64_t z = v / MN8;
        const int64_t r = v - z * MN8;
        int m, n;
        float vals[8];
        if (g.c.contig_n) {
            const int nv = g.N / 8;
            m = (int)(r / nv); n = (int)(r % nv) * 8;
            V8<float>::load(g.split_ws + (z * g.M + m) * (int64_t)g.N + n, vals);
            for (int s = 1; s < g.splits; ++s) {
                float t[8];
                V8<float>::load(g.split_ws + s * plane + (z * g.M + m) * (int64_t)g.N + n, t);
#pragma unroll
                for (int q = 0; q < 8; ++q) vals[q] += t[q];
            }
        } else {
            const int mv = g.M / 8;
            n = (int)(r / mv); m = (int)(r % mv) * 8;
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                float acc = 0.f;
                for (int s = 0; s < g.splits; ++s) acc += g.split_ws[s * plane + (z * g.M + m + q) * (int64_t)g.N + n];
                vals[q] = acc;
            }
        }
#pragma unroll
        for (int q = 0; q < 8; ++q) vals[q] *= g.c.alpha;
        int dummy = 0;
        store_vec<T>(g, map_off(g.c.batch, (uint32_t)z, 1, &dummy), m, n, vals);
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

// Float32 contractions on v_mfma_f32_32x32x2f32: a 64x64 block tile, four
// waves of 32x32, k-steps of 16 staged through LDS (operands gathered
// element by element through their index maps, so every layout and ragged
// size is taken; zeros past M, N, K), fp32 products and accumulation.  Lane
// l of a 32x32x2 step supplies row l % 32 of A and column l % 32 of B at
// k = 2 s + l / 32; the result's lane l holds column l % 32 at rows
// 8 (r / 4) + 4 (l / 32) + r % 4.  The epilogue stores element by element
// through the output maps (bias, residual, segments as in the 16-bit path).
constexpr int F32_T = 64, F32_K = 16;

__global__ __launch_bounds__(256) void gemm_f32(GemmArgs g) {
    __shared__ float sa[F32_K][F32_T + 1];
    __shared__ float sb[F32_K][F32_T + 1];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int m0 = (blockIdx.y % g.tiles_m) * F32_T, n0 = blockIdx.x * F32_T;
    const uint32_t z = blockIdx.y / g.tiles_m;
    int dummy = 0;
    const int64_t aoff = map_off(g.a.batch, z, 1, &dummy);
    const int64_t boff = map_off(g.b.batch, z, 1, &dummy);
    floatx16 acc;
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[r] = 0.f;
    for (int k0 = 0; k0 < g.K; k0 += F32_K) {
        // each thread gathers 4 elements of each operand tile
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int idx = u * 256 + tid, kk = idx / F32_T, o = idx % F32_T;
            const int k = k0 + kk;
            sa[kk][o] = (m0 + o < g.M && k < g.K) ? op_elem(g.a, aoff, m0 + o, k) : 0.f;
            sb[kk][o] = (n0 + o < g.N && k < g.K) ? op_elem(g.b, boff, n0 + o, k) : 0.f;
        }
        __syncthreads();
#pragma unroll
        for (int s2 = 0; s2 < F32_K / 2; ++s2) {
            const int k = 2 * s2 + (lane >> 5);
            acc = __builtin_amdgcn_mfma_f32_32x32x2f32(sa[k][wm * 32 + (lane & 31)], sb[k][wn * 32 + (lane & 31)],
                                                       acc, 0, 0, 0);
        }
        __syncthreads();
    }
    const Epilogue& e = g.c;
    const int n = n0 + wn * 32 + (lane & 31);
    if (n >= g.N) return;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        const int m = m0 + wm * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        if (m >= g.M) continue;
        float v = acc[r] * e.alpha;
        if (e.bias[0]) {
            int bseg = 0;
            const int64_t bo = map_off(e.bias_map, (uint32_t)(e.bias_on_m ? m : n), e.bias_nseg, &bseg);
            v += reinterpret_cast<const float*>(seg_ptr(e.bias, bseg))[bo];
        }
        int sm = 0, sn = 0;
        const int64_t off = map_off(e.batch, z, 1, &dummy) +
                            map_off(e.mmap, (uint32_t)m, e.seg_on_m ? e.nseg : 1, &sm) +
                            map_off(e.nmap, (uint32_t)n, e.seg_on_m ? 1 : e.nseg, &sn);
        const int seg = e.seg_on_m ? sm : sn;
        if (e.resid) v += reinterpret_cast<const float*>(e.resid)[off];
        reinterpret_cast<float*>(seg_ptr(e.ptr, seg))[off] = v;
    }
}

// Tile configurations: (BM, BN, waves along m, waves along n).
struct TileCfg {
    int bm, bn, wgm, wgn;
};
// 0-4: register-staged kernel; 5-8: asynchronous (global -> LDS) kernel;
// 9-12: asynchronous kernel on 32x32x16 MFMAs; 13: lean 256x256 kernel
// (8 waves of 128x64, four stages of 32-wide k-steps); 14: the general
// 256x256 kernel with the same waves; 15: lean 128x128 kernel (8 waves of
// 64x32, four stages of 64-wide k-steps); 16: lean 128x128 kernel with two
// k groups of 4 waves of 64x64.  Contractions a lean kernel does not take
// run on 14 (for 13) or 11 (for 15, 16).  17: lean 256x256 kernel with 4
// waves of 128x128 (one per SIMD); 18: lean 128x128 kernel with 4 waves of
// 64x64 (one per SIMD): each SIMD's wave then reads every fragment of its
// region once per k-step, where two waves per SIMD read the shared operand
// twice.  Contractions they do not take run on 14 (17) or 11 (18).
// 19: lean 256x192 kernel (4 waves of 128x96) for outputs whose width is a
// multiple of 192 but leaves 256x256 tiles short of the CU count (3072
// columns: 16 x 16 tiles instead of 16 x 12); the 192-wide operand must be
// contiguous along k (else run as 13).  20, 21, 22: the tiles of 17, 19
// and 18 with the interleaved schedule (each MFMA issued next to its share
// of the fragment reads and copies); contractions they do not take run as
// 17, 19 and 18 would.  23, 24: the tile and waves of 13 with the
// ping-pong schedule (the two wave rows alternate between reading a
// k-step's fragments and multiplying them), four and five stages (copies
// two and three k-steps ahead); contractions they do not take run as 13
// would.  25: the ping-pong schedule on a 256x192 tile of 8 waves of 64x96
// (4 wave rows, 2 columns), for a B operand contiguous along k (otherwise
// run as 23): 3072-wide outputs get 16 x 16 tiles, every CU one.
constexpr TileCfg CFGS[] = {{256, 256, 2, 4}, {256, 128, 2, 2}, {128, 128, 2, 2}, {256, 64, 4, 1}, {128, 64, 2, 2},
                            {256, 128, 2, 2}, {128, 128, 2, 2}, {256, 64, 4, 1}, {128, 64, 2, 2},
                            {256, 256, 2, 4}, {256, 128, 2, 2}, {128, 128, 2, 2}, {256, 128, 4, 2},
                            {256, 256, 2, 4}, {256, 256, 2, 4}, {128, 128, 2, 4}, {128, 128, 2, 2},
                            {256, 256, 2, 2}, {128, 128, 2, 2}, {256, 192, 2, 2}, {256, 256, 2, 2}, {256, 192, 2, 2}, {128, 128, 2, 2},
                            {256, 256, 2, 4}, {256, 256, 2, 4}, {256, 192, 4, 2}};
static_assert(sizeof(CFGS) / sizeof(CFGS[0]) == GEMM_MAX_CFG + 1, "configuration table");
constexpr int NCFG = sizeof(CFGS) / sizeof(CFGS[0]);

template <typename T, int BM, int BN, int WGM, int WGN, int DEPTH>
void launch_cfg(const GemmArgs& g, hipStream_t st) {
    dim3 grid(g.tiles_m * g.tiles_n, g.batch * (g.splits > 1 ? g.splits : 1));
    dim3 block(64 * WGM * WGN);
    if (g.a.kcontig && g.b.kcontig)
        hipLaunchKernelGGL((gemm_mfma<T, BM, BN, WGM, WGN, DEPTH, true, true>), grid, block, 0, st, g);
    else if (g.a.kcontig)
        hipLaunchKernelGGL((gemm_mfma<T, BM, BN, WGM, WGN, DEPTH, true, false>), grid, block, 0, st, g);
    else if (g.b.kcontig)
        hipLaunchKernelGGL((gemm_mfma<T, BM, BN, WGM, WGN, DEPTH, false, true>), grid, block, 0, st, g);
    else
        hipLaunchKernelGGL((gemm_mfma<T, BM, BN, WGM, WGN, DEPTH, false, false>), grid, block, 0, st, g);
}

template <typename T, int BM, int BN, int WGM, int WGN>
void launch_dma(const GemmArgs& g, hipStream_t st) {
    dim3 grid(g.tiles_m * g.tiles_n, g.batch * (g.splits > 1 ? g.splits : 1));
    dim3 block(64 * WGM * WGN);
    if (g.a.kcontig && g.b.kcontig)
        hipLaunchKernelGGL((gemm_dma<T, BM, BN, WGM, WGN, true, true>), grid, block, 0, st, g);
    else if (g.a.kcontig)
        hipLaunchKernelGGL((gemm_dma<T, BM, BN, WGM, WGN, true, false>), grid, block, 0, st, g);
    else if (g.b.kcontig)
        hipLaunchKernelGGL((gemm_dma<T, BM, BN, WGM, WGN, false, true>), grid, block, 0, st, g);
    else
        hipLaunchKernelGGL((gemm_dma<T, BM, BN, WGM, WGN, false, false>), grid, block, 0, st, g);
}

template <typename T, int BM, int BN, int WGM, int WGN, int STAGES>
void launch_x32(const GemmArgs& g, hipStream_t st) {
    dim3 grid(g.tiles_m * g.tiles_n, g.batch * (g.splits > 1 ? g.splits : 1));
    dim3 block(64 * WGM * WGN);
    if (g.a.kcontig && g.b.kcontig)
        hipLaunchKernelGGL((gemm_x32<T, BM, BN, WGM, WGN, STAGES, true, true>), grid, block, 0, st, g);
    else if (g.a.kcontig)
        hipLaunchKernelGGL((gemm_x32<T, BM, BN, WGM, WGN, STAGES, true, false>), grid, block, 0, st, g);
    else if (g.b.kcontig)
        hipLaunchKernelGGL((gemm_x32<T, BM, BN, WGM, WGN, STAGES, false, true>), grid, block, 0, st, g);
    else
        hipLaunchKernelGGL((gemm_x32<T, BM, BN, WGM, WGN, STAGES, false, false>), grid, block, 0, st, g);
}

template <typename T, int BM, int BN, int WGM, int WGN, int BKS, int STAGES, int KG = 1, bool RS = false>
void launch_lean(const GemmArgs& g, hipStream_t st) {
    dim3 grid(g.tiles_m * g.tiles_n, g.batch * (g.splits > 1 ? g.splits : 1));
    dim3 block(64 * WGM * WGN * KG);
    if constexpr (RS) {
        // row sums are produced for an outer-contiguous A only
        if (g.b.kcontig)
            hipLaunchKernelGGL((gemm_lean<T, BM, BN, WGM, WGN, BKS, STAGES, false, true, KG, true>), grid, block, 0,
                               st, g);
        else
            hipLaunchKernelGGL((gemm_lean<T, BM, BN, WGM, WGN, BKS, STAGES, false, false, KG, true>), grid, block, 0,
                               st, g);
        return;
    }
    if (g.a.kcontig && g.b.kcontig)
        hipLaunchKernelGGL((gemm_lean<T, BM, BN, WGM, WGN, BKS, STAGES, true, true, KG>), grid, block, 0, st, g);
    else if (g.a.kcontig)
        hipLaunchKernelGGL((gemm_lean<T, BM, BN, WGM, WGN, BKS, STAGES, true, false, KG>), grid, block, 0, st, g);
    else if (g.b.kcontig)
        hipLaunchKernelGGL((gemm_lean<T, BM, BN, WGM, WGN, BKS, STAGES, false, true, KG>), grid, block, 0, st, g);
    else
        hipLaunchKernelGGL((gemm_lean<T, BM, BN, WGM, WGN, BKS, STAGES, false, false, KG>), grid, block, 0, st, g);
}

// Lean kernels with the activation step in the epilogue (the operand
// layouts settle_act admits: mode 1 A and B contiguous along k, mode 2 A
// contiguous along k, B along n).
template <typename T, int BM, int BN, int WGM, int WGN, int BKS, int STAGES>
void launch_lean_act(const GemmArgs& g, hipStream_t st) {
    dim3 grid(g.tiles_m * g.tiles_n, g.batch);
    dim3 block(64 * WGM * WGN);
    if (g.c.act_mode == 1)
        hipLaunchKernelGGL((gemm_lean<T, BM, BN, WGM, WGN, BKS, STAGES, true, true, 1, false, 0, 1>), grid, block,
                           0, st, g);
    else
        hipLaunchKernelGGL((gemm_lean<T, BM, BN, WGM, WGN, BKS, STAGES, true, false, 1, false, 0, 2>), grid,
                           block, 0, st, g);
}

// Lean kernels with the interleaved one-wave-per-SIMD schedule.
template <typename T, int BM, int BN, int WGM, int WGN, int BKS, int STAGES>
void launch_lean_il(const GemmArgs& g, hipStream_t st) {
    dim3 grid(g.tiles_m * g.tiles_n, g.batch * (g.splits > 1 ? g.splits : 1));
    dim3 block(64 * WGM * WGN);
    if (g.a.kcontig && g.b.kcontig)
        hipLaunchKernelGGL((gemm_lean<T, BM, BN, WGM, WGN, BKS, STAGES, true, true, 1, false, 1>), grid, block, 0,
                           st, g);
    else if (g.a.kcontig)
        hipLaunchKernelGGL((gemm_lean<T, BM, BN, WGM, WGN, BKS, STAGES, true, false, 1, false, 1>), grid, block, 0,
                           st, g);
    else if (g.b.kcontig)
        hipLaunchKernelGGL((gemm_lean<T, BM, BN, WGM, WGN, BKS, STAGES, false, true, 1, false, 1>), grid, block, 0,
                           st, g);
    else
        hipLaunchKernelGGL((gemm_lean<T, BM, BN, WGM, WGN, BKS, STAGES, false, false, 1, false, 1>), grid, block,
                           0, st, g);
}

template <typename T, int BM, int BN, int WGM, int WGN, int BKS, int STAGES>
void launch_lean_il_bk(const GemmArgs& g, hipStream_t st) {
    dim3 grid(g.tiles_m * g.tiles_n, g.batch * (g.splits > 1 ? g.splits : 1));
    dim3 block(64 * WGM * WGN);
    if (g.a.kcontig)
        hipLaunchKernelGGL((gemm_lean<T, BM, BN, WGM, WGN, BKS, STAGES, true, true, 1, false, 1>), grid, block, 0,
                           st, g);
    else
        hipLaunchKernelGGL((gemm_lean<T, BM, BN, WGM, WGN, BKS, STAGES, false, true, 1, false, 1>), grid, block, 0,
                           st, g);
}

// Lean kernels with the ping-pong schedule (two wave rows alternating
// between fragment reads and MFMAs), also with the activation epilogues.
template <typename T, int BM, int BN, int WGM, int WGN, int BKS, int STAGES>
void launch_lean_pp(const GemmArgs& g, hipStream_t st) {
    dim3 grid(g.tiles_m * g.tiles_n, g.batch * (g.splits > 1 ? g.splits : 1));
    dim3 block(64 * WGM * WGN);
    if (g.c.act_mode == 1)
        hipLaunchKernelGGL((gemm_lean<T, BM, BN, WGM, WGN, BKS, STAGES, true, true, 1, false, 2, 1>), grid, block,
                           0, st, g);
    else if (g.c.act_mode == 2)
        hipLaunchKernelGGL((gemm_lean<T, BM, BN, WGM, WGN, BKS, STAGES, true, false, 1, false, 2, 2>), grid,
                           block, 0, st, g);
    else if (g.a.kcontig && g.b.kcontig)
        hipLaunchKernelGGL((gemm_lean<T, BM, BN, WGM, WGN, BKS, STAGES, true, true, 1, false, 2>), grid, block, 0,
                           st, g);
    else if (g.a.kcontig)
        hipLaunchKernelGGL((gemm_lean<T, BM, BN, WGM, WGN, BKS, STAGES, true, false, 1, false, 2>), grid, block, 0,
                           st, g);
    else if (g.b.kcontig)
        hipLaunchKernelGGL((gemm_lean<T, BM, BN, WGM, WGN, BKS, STAGES, false, true, 1, false, 2>), grid, block, 0,
                           st, g);
    else
        hipLaunchKernelGGL((gemm_lean<T, BM, BN, WGM, WGN, BKS, STAGES, false, false, 1, false, 2>), grid, block,
                           0, st, g);
}

// Ping-pong kernels whose B tile width only suits a k-contiguous B operand.
template <typename T, int BM, int BN, int WGM, int WGN, int BKS, int STAGES>
void launch_lean_pp_bk(const GemmArgs& g, hipStream_t st) {
    dim3 grid(g.tiles_m * g.tiles_n, g.batch * (g.splits > 1 ? g.splits : 1));
    dim3 block(64 * WGM * WGN);
    if (g.c.act_mode == 1)
        hipLaunchKernelGGL((gemm_lean<T, BM, BN, WGM, WGN, BKS, STAGES, true, true, 1, false, 2, 1>), grid, block,
                           0, st, g);
    else if (g.a.kcontig)
        hipLaunchKernelGGL((gemm_lean<T, BM, BN, WGM, WGN, BKS, STAGES, true, true, 1, false, 2>), grid, block, 0,
                           st, g);
    else
        hipLaunchKernelGGL((gemm_lean<T, BM, BN, WGM, WGN, BKS, STAGES, false, true, 1, false, 2>), grid, block, 0,
                           st, g);
}

// Lean kernels whose B tile width only suits a k-contiguous B operand.
template <typename T, int BM, int BN, int WGM, int WGN, int BKS, int STAGES>
void launch_lean_bk(const GemmArgs& g, hipStream_t st) {
    dim3 grid(g.tiles_m * g.tiles_n, g.batch * (g.splits > 1 ? g.splits : 1));
    dim3 block(64 * WGM * WGN);
    if (g.a.kcontig)
        hipLaunchKernelGGL((gemm_lean<T, BM, BN, WGM, WGN, BKS, STAGES, true, true, 1>), grid, block, 0, st, g);
    else
        hipLaunchKernelGGL((gemm_lean<T, BM, BN, WGM, WGN, BKS, STAGES, false, true, 1>), grid, block, 0, st, g);
}

template <typename T, int BM, int BN, int WGM, int WGN, int BKS, int STAGES>
void launch_lean_pair(const GemmArgs& g0, const GemmArgs& g1, hipStream_t st) {
    dim3 grid(g0.tiles_m * g0.tiles_n + g1.tiles_m * g1.tiles_n);
    dim3 block(64 * WGM * WGN);
    if (g0.c.rsum) {
        // row sums of g0's A (outer-contiguous) are produced
        if (g0.b.kcontig)
            hipLaunchKernelGGL((gemm_lean_pair<T, BM, BN, WGM, WGN, BKS, STAGES, false, true, true>), grid, block, 0,
                               st, g0, g1);
        else
            hipLaunchKernelGGL((gemm_lean_pair<T, BM, BN, WGM, WGN, BKS, STAGES, false, false, true>), grid, block,
                               0, st, g0, g1);
        return;
    }
    if (g0.a.kcontig && g0.b.kcontig)
        hipLaunchKernelGGL((gemm_lean_pair<T, BM, BN, WGM, WGN, BKS, STAGES, true, true>), grid, block, 0, st, g0, g1);
    else if (g0.a.kcontig)
        hipLaunchKernelGGL((gemm_lean_pair<T, BM, BN, WGM, WGN, BKS, STAGES, true, false>), grid, block, 0, st, g0, g1);
    else if (g0.b.kcontig)
        hipLaunchKernelGGL((gemm_lean_pair<T, BM, BN, WGM, WGN, BKS, STAGES, false, true>), grid, block, 0, st, g0, g1);
    else
        hipLaunchKernelGGL((gemm_lean_pair<T, BM, BN, WGM, WGN, BKS, STAGES, false, false>), grid, block, 0, st, g0, g1);
}

template <typename T, int WGM, int WGN>
void launch_big(const GemmArgs& g, hipStream_t st) {
    dim3 grid(g.tiles_m * g.tiles_n, g.batch * (g.splits > 1 ? g.splits : 1));
    dim3 block(64 * WGM * WGN);
    if (g.a.kcontig && g.b.kcontig) hipLaunchKernelGGL((gemm_big<T, WGM, WGN, true, true>), grid, block, 0, st, g);
    else if (g.a.kcontig) hipLaunchKernelGGL((gemm_big<T, WGM, WGN, true, false>), grid, block, 0, st, g);
    else if (g.b.kcontig) hipLaunchKernelGGL((gemm_big<T, WGM, WGN, false, true>), grid, block, 0, st, g);
    else hipLaunchKernelGGL((gemm_big<T, WGM, WGN, false, false>), grid, block, 0, st, g);
}

template <typename T>
void launch_t(const GemmArgs& g, hipStream_t st) {
    switch (g.cfg) {
        case 13:
            if (g.c.rsum) launch_lean<T, 256, 256, 2, 4, 32, 4, 1, true>(g, st);
            else if (g.c.act_mode) launch_lean_act<T, 256, 256, 2, 4, 32, 4>(g, st);
            else launch_lean<T, 256, 256, 2, 4, 32, 4>(g, st);
            break;
        case 15:
            if (g.c.rsum) launch_lean<T, 128, 128, 2, 4, 64, 4, 1, true>(g, st);
            else if (g.c.act_mode) launch_lean_act<T, 128, 128, 2, 4, 64, 4>(g, st);
            else launch_lean<T, 128, 128, 2, 4, 64, 4>(g, st);
            break;
        case 16: launch_lean<T, 128, 128, 2, 2, 64, 4, 2>(g, st); break;
        case 17: launch_lean<T, 256, 256, 2, 2, 32, 4>(g, st); break;
        case 18: launch_lean<T, 128, 128, 2, 2, 64, 4>(g, st); break;
        case 19: launch_lean_bk<T, 256, 192, 2, 2, 32, 4>(g, st); break;
        case 20: launch_lean_il<T, 256, 256, 2, 2, 32, 4>(g, st); break;
        case 21: launch_lean_il_bk<T, 256, 192, 2, 2, 32, 4>(g, st); break;
        case 22: launch_lean_il<T, 128, 128, 2, 2, 64, 4>(g, st); break;
        case 23: launch_lean_pp<T, 256, 256, 2, 4, 32, 4>(g, st); break;
        case 24: launch_lean_pp<T, 256, 256, 2, 4, 32, 5>(g, st); break;
        case 25: launch_lean_pp_bk<T, 256, 192, 4, 2, 32, 4>(g, st); break;
        case 14: launch_big<T, 2, 4>(g, st); break;
        case 9: launch_x32<T, 256, 256, 2, 4, 2>(g, st); break;
        case 10: launch_x32<T, 256, 128, 2, 2, 3>(g, st); break;
        case 11: launch_x32<T, 128, 128, 2, 2, 4>(g, st); break;
        case 12: launch_x32<T, 256, 128, 4, 2, 3>(g, st); break;
        case 5: launch_dma<T, 256, 128, 2, 2>(g, st); break;
        case 6: launch_dma<T, 128, 128, 2, 2>(g, st); break;
        case 7: launch_dma<T, 256, 64, 4, 1>(g, st); break;
        case 8: launch_dma<T, 128, 64, 2, 2>(g, st); break;
        case 0: launch_cfg<T, 256, 256, 2, 4, 1>(g, st); break;
        case 1: launch_cfg<T, 256, 128, 2, 2, 1>(g, st); break;
        case 2: launch_cfg<T, 128, 128, 2, 2, 1>(g, st); break;
        case 3: launch_cfg<T, 256, 64, 4, 1, 1>(g, st); break;
        default: launch_cfg<T, 128, 64, 2, 2, 1>(g, st); break;
    }
    if (g.splits > 1) {
        trace_next("reduce");
        const int64_t total = (int64_t)g.batch * g.M * g.N / 8;
        int64_t blocks = (total + 255) / 256;
        if (blocks > 4096) blocks = 4096;
        hipLaunchKernelGGL((splitk_reduce<T>), dim3((unsigned)blocks), dim3(256), 0, st, g);
    }
}

int64_t ntiles(const TileCfg& c, const GemmArgs& g) {
    return (int64_t)((g.M + c.bm - 1) / c.bm) * ((g.N + c.bn - 1) / c.bn) * g.batch;
}

// Tile and split choice, from measurements of the layer's contraction
// shapes on MI355X (every configuration x split 1/2/4): the lean 256x256
// kernel (ping-pong schedule) when that tile alone gives (nearly) every CU
// a block; otherwise the
// lean 128x128 kernel, split along k for long-k contractions with few
// output tiles (up to four ways, towards one block per CU); narrow outputs
// (n <= 64) on the asynchronous 128x64 tile.  A lean kernel hands
// contractions it does not take to its general counterpart.  Explicit
// choices (cfg >= 0, splits > 0) are kept.
void choose(GemmArgs& g) {
    constexpr int64_t CUS = 256;
    const bool split_ok = g.split_ws != nullptr && g.batch == 1;
    int want_split = 1;
    if (g.cfg < 0 || g.cfg >= NCFG) {
        if (g.N <= 64) {
            g.cfg = 8;
        } else if (ntiles(CFGS[13], g) * 4 >= CUS * 3) {
            // (the 256x192 tiles of cfg 19, which give 3072-wide outputs
            // every CU where 256x256 leaves a quarter idle, measured slower
            // than cfg 13 with its two waves per SIMD; a plan may still pick
            // them).  The ping-pong schedule (cfg 23) runs the k-loop about
            // 10 % faster than cfg 13 at the same fixed cost; row sums are
            // produced by cfg 13 only.
            g.cfg = g.c.rsum ? 13 : 23;
            // a 192-wide tile where 256-wide ones leave CUs idle and 192-wide
            // ones still fit in one round (3072-wide outputs: 256 against
            // 192 tiles)
            if (!g.c.rsum && g.c.act_mode != 2 && g.b.kcontig && g.N % 192 == 0 && ntiles(CFGS[23], g) < CUS &&
                ntiles(CFGS[25], g) <= CUS)
                g.cfg = 25;
        } else {
            g.cfg = 15;
            const int64_t t = ntiles(CFGS[15], g);
            if (split_ok && g.K >= 2048 && t < CUS * 3 / 4) want_split = (int)std::min<int64_t>(4, std::max<int64_t>(1, CUS / t));
        }
    }
    // the 32x32x16 kernels' epilogues take no bias along m and only output
    // maps affine over 32-wide blocks; of them only the lean 128x128 kernel
    // takes a residual operand
    if (((g.c.bias[0] && g.c.bias_on_m) || !g.blk32) && g.cfg >= 9) g.cfg = 8;
    if (g.c.resid && g.cfg >= 9 && g.cfg != 15 && g.cfg != 16 && g.cfg != 18 && g.cfg != 22) g.cfg = 8;
    if (g.splits <= 0) {
        int s = split_ok ? want_split : 1;
        while (s > 1 && (g.K / s < 256 || (int64_t)s * g.batch * g.M * g.N > g.split_cap)) --s;
        g.splits = s;
    }
    if (g.splits > 1) {
        const int ksteps = (g.K + BK - 1) / BK;
        g.kper = (ksteps + g.splits - 1) / g.splits * BK;
        g.splits = (g.K + g.kper - 1) / g.kper;
    }
    if (g.cfg == 19 && !g.b.kcontig) g.cfg = 13;
    if (g.cfg == 21 && !g.b.kcontig) g.cfg = 20;
    if (g.cfg == 25 && !g.b.kcontig) g.cfg = 23;
    if ((g.cfg == 13 || g.cfg == 17 || g.cfg == 19 || g.cfg == 20 || g.cfg == 21 || g.cfg == 23 || g.cfg == 24 ||
         g.cfg == 25) &&
        !lean_ok(g, 32))
        g.cfg = 14;
    if ((g.cfg == 15 || g.cfg == 16 || g.cfg == 18 || g.cfg == 22) && !lean_ok(g, 64)) g.cfg = g.c.resid ? 8 : 11;
    // tile counts of the configuration that runs (the fallback from 15 to 8
    // changes the tile width)
    const TileCfg& c = CFGS[g.cfg];
    g.tiles_m = (g.M + c.bm - 1) / c.bm;
    g.tiles_n = (g.N + c.bn - 1) / c.bn;
}

// Classifies the output addressing for the fast store pass.
void set_affine(GemmArgs& g) {
    const Epilogue& e = g.c;
    const bool cn = e.contig_n != 0;
    g.blk32 = block32_linear(e.mmap) && block32_linear(e.nmap);
    g.affine = 0;
    g.bias_mode = 0;
    g.ldc = 0;
    if (e.nseg != 1 || e.mmap.r0 != 0 || e.nmap.r0 != 0) return;
    if (cn ? e.nmap.s0 != 1 : e.mmap.s0 != 1) return;
    if (e.bias[0]) {
        if (e.bias_nseg != 1 || e.bias_map.r0 != 0 || e.bias_map.s0 != 1) return;
        g.bias_mode = (e.bias_on_m != 0) == !cn ? 1 : 2;
    }
    g.ldc = cn ? e.mmap.s0 : e.nmap.s0;
    g.affine = 1;
}

// Whether the lean kernels may stage the output (and split partials)
// through LDS: row-major single-pointer output without a residual, 16-byte
// aligned rows of whole 8-element pieces.
void set_ep_stage(GemmArgs& g) {
    const Epilogue& e = g.c;
    g.ep_stage = 0;
    if (g.N % 8) return;
    if ((uintptr_t)g.split_ws % 16 == 0) g.ep_stage |= 2;
    const bool bias_ok = !e.bias[0] || g.bias_mode == 1;
    if (g.affine && e.contig_n && !e.resid && bias_ok && g.ldc % 8 == 0 && (g.batch == 1 || e.batch.s0 % 8 == 0) &&
        e.batch.r0 == 0 && ((uintptr_t)e.ptr[0] % 16) == 0) {
        g.ep_stage |= 1;
        return;
    }
    // an output through index maps (head permutation, segments): staged
    // when every aligned 8-column piece of a row is 8 contiguous elements
    // at a 16-byte aligned address
    auto mult8 = [](int64_t v) { return v % 8 == 0; };
    bool ok = e.contig_n && !e.resid && !(e.bias[0] && e.bias_on_m) && e.nmap.s0 == 1 &&
              (e.nmap.r0 == 0 || e.nmap.r0 % 8 == 0) && mult8(e.nmap.s1) && mult8(e.nmap.s2) &&
              mult8(e.mmap.s0) && mult8(e.mmap.s1) && mult8(e.mmap.s2) && mult8(e.batch.s0) &&
              mult8(e.batch.s1) && mult8(e.batch.s2);
    for (int i = 0; i < (e.nseg > 0 ? e.nseg : 1); ++i) ok = ok && e.ptr[i] && ((uintptr_t)e.ptr[i] % 16) == 0;
    if (ok) g.ep_stage |= 4;
}

// The plan of the running call (entries keyed by sizes, dtype and operand
// contiguity) and this thread's launch record.
thread_local const dm_plan* t_plan = nullptr;
thread_local bool t_log_on = false;
thread_local std::vector<dm_contract_choice> t_log;

bool same_contraction(const dm_contract_choice& e, const GemmArgs& g, int dtype) {
    return e.M == g.M && e.N == g.N && e.K == g.K && e.batch == g.batch && e.dtype == dtype &&
           e.a_kcontig == (g.a.kcontig ? 1 : 0) && e.b_kcontig == (g.b.kcontig ? 1 : 0);
}

// A plan entry's tile and split factor for an automatically configured
// contraction; the split factor is cut to what the scratch holds.
void apply_plan(GemmArgs& g, int dtype) {
    if (!t_plan) return;
    for (const dm_contract_choice& e : t_plan->entries) {
        if (!same_contraction(e, g, dtype)) continue;
        g.cfg = e.tile_cfg;
        int s = e.splits > 1 ? e.splits : 1;
        if (!g.split_ws || g.batch != 1) s = 1;
        while (s > 1 && (g.K / s < 256 || (int64_t)s * g.batch * g.M * g.N > g.split_cap)) --s;
        g.splits = s;
        return;
    }
}

// Keeps the activation step only where the staged epilogue takes it:
// unsplit lean 256x256 or 128x128 kernel of 8 waves (2 wave rows: cfg 13,
// 15 and the ping-pong forms of 13, 23 and 24; mode 1 also on the 256x192
// ping-pong tile, cfg 25), staged
// row-major output, 16-bit storage, no alpha scaling or bias; mode 1 with A
// and B contiguous along k, mode 2 with A contiguous along k and B along
// n, its partial rows (2 per tile row) within act_part_cap.  Returns the
// partial rows mode 2 writes (1 for mode 1), 0 when not taken.
int settle_act(GemmArgs& g, int dtype) {
    const Epilogue& e = g.c;
    // (cfg 25, 4 wave rows and 96-column waves, takes mode 1 only: mode 2's
    // partial rows assume 2 wave rows and its column groups a power-of-two
    // lane count)
    const bool tile_ok = g.cfg == 13 || g.cfg == 15 || g.cfg == 23 || g.cfg == 24 || (g.cfg == 25 && e.act_mode == 1);
    bool ok = e.act_mode && dtype != G_F32 && tile_ok && !e.rsum && g.splits <= 1 &&
              (g.ep_stage & 1) && !e.out_f32 && !e.bias[0] && e.alpha == 1.0f && e.act_bias && g.batch == 1;
    int parts = 1;
    if (ok && e.act_mode == 1) ok = g.a.kcontig && g.b.kcontig && e.act_out && ((uintptr_t)e.act_out % 16) == 0;
    else if (ok && e.act_mode == 2) {
        parts = g.tiles_m * 2;
        ok = g.a.kcontig && !g.b.kcontig && e.act_in && e.act_part && parts <= e.act_part_cap &&
             ((uintptr_t)e.act_in % 16) == 0 && ((uintptr_t)e.act_part % 16) == 0;
    } else {
        ok = false;
    }
    if (!ok) g.c.act_mode = 0;
    return ok ? parts : 0;
}

thread_local int t_act_parts = 0;

thread_local int t_rsum_parts = 0;

// Keeps the row-sum request only where the kernel that runs produces it
// (the lean 256x256 and 128x128 tiles, both 4 wave tiles wide, unsplit, A
// outer-contiguous) and its partial rows fit.
void settle_rowsums(GemmArgs& g) {
    constexpr int WGN = 4;
    const bool lean1 = g.cfg == 13 || g.cfg == 15;
    const int nw = g.tiles_n * WGN;
    const bool ok = g.c.rsum != nullptr && lean1 && g.splits <= 1 && !g.a.kcontig && g.batch == 1 &&
                    nw <= g.c.rsum_cap && g.c.rsum_ld >= g.M;
    t_rsum_parts = ok ? nw : 0;
    if (!ok) g.c.rsum = nullptr;
}

void log_launch(const GemmArgs& g, int dtype) {
    if (!t_log_on) return;
    dm_contract_choice r{};
    r.M = g.M; r.N = g.N; r.K = g.K; r.batch = g.batch; r.dtype = dtype;
    r.a_kcontig = g.a.kcontig ? 1 : 0; r.b_kcontig = g.b.kcontig ? 1 : 0;
    r.tile_cfg = g.cfg; r.splits = g.splits > 1 ? g.splits : 1;
    strncpy(r.label, trace_current_label(), sizeof(r.label) - 1);
    t_log.push_back(r);
}

}  // namespace

const dm_plan* current_plan() { return t_plan; }
int gemm_rowsum_parts() { return t_rsum_parts; }

static int prepare(GemmArgs& g, int dtype, bool pair);

bool gemm_act_fusable(int dtype, const GemmArgs& args) {
    if (dtype == G_F32 || args.M <= 0 || args.N <= 0 || args.K <= 0 || args.batch != 1) return false;
    GemmArgs g = args;
    if (prepare(g, dtype, false)) return false;
    return settle_act(g, dtype) > 0;
}

int gemm_act_parts() { return t_act_parts; }
PlanScope::PlanScope(const dm_plan* p) : prev(t_plan) { t_plan = p; }
PlanScope::~PlanScope() { t_plan = prev; }
int current_attn_path() { return t_plan ? t_plan->attn_path : 0; }

FusedLayout fused_layout(int dtype, int64_t T, int I, int F) {
    (void)F;
    FusedLayout f{};
    const dm_layout_choice c = t_plan ? t_plan->layout : dm_layout_choice{-1, -1, -1, -1};
    f.ln_form = c.ln_bwd_form > 0 ? c.ln_bwd_form : 0;
    f.ln_lanes = c.ln_lanes > 0 ? c.ln_lanes : 0;
    f.dO_t = ln_bwd_uses_split(I, dtype, f.ln_form) && c.dO_transposed != 0;
    f.dH_t = dtype != DM_F32 && T % 8 == 0 && c.dH_transposed == 1;
    return f;
}

void plan_log_set(bool on) {
    t_log_on = on;
    if (on) t_log.clear();
}

int plan_log_copy(dm_contract_choice* out, int cap) {
    for (int i = 0; i < cap && i < (int)t_log.size(); ++i) out[i] = t_log[i];
    return (int)t_log.size();
}

// Validation, plan and configuration of a 16-bit contraction; `pair`: when
// no plan entry fixes the configuration, ask for the lean 128x128 kernel
// unsplit (what a paired launch runs).
static int prepare(GemmArgs& g, int dtype, bool pair) {
    if (g.K % 8 || g.M % 8 || g.N % 8)
        return set_error(DM_ERR_UNSUPPORTED, "contraction sizes must be multiples of 8");
    if (g.c.bias[0] && ((g.c.bias_on_m != 0) == (g.c.contig_n == 0)) && g.c.bias_map.r0 % 8 != 0)
        return set_error(DM_ERR_UNSUPPORTED, "bias map radix along the output vector must be a multiple of 8");
    if (!g.split_ws) g.splits = 1;
    set_affine(g);
    set_ep_stage(g);
    if (g.cfg < 0) apply_plan(g, dtype);
    if (pair && g.cfg < 0) { g.cfg = 15; g.splits = 1; }
    choose(g);
    if (g.splits > 1 && (int64_t)g.splits * g.batch * g.M * g.N > g.split_cap)
        return set_error(DM_ERR_WORKSPACE, "split-k scratch too small");
    if ((int64_t)g.batch * g.splits > 65535) return set_error(DM_ERR_UNSUPPORTED, "contraction grid too large");
    return 0;
}

int launch_gemm(int dtype, const GemmArgs& args, hipStream_t st) {
    t_rsum_parts = 0;
    t_act_parts = 0;
    GemmArgs g = args;
    if (g.M <= 0 || g.N <= 0 || g.batch <= 0) return 0;
    if (g.K <= 0) return set_error(DM_ERR_ARG, "contraction with K <= 0");
    if (g.batch > 65535) return set_error(DM_ERR_UNSUPPORTED, "contraction batch above 65535");
    if (dtype == G_F32) {
        g.tiles_m = (g.M + F32_T - 1) / F32_T;
        g.tiles_n = (g.N + F32_T - 1) / F32_T;
        if ((int64_t)g.tiles_m * g.batch > 65535)
            return set_error(DM_ERR_UNSUPPORTED, "fp32 contraction grid too large");
        dim3 grid(g.tiles_n, g.tiles_m * g.batch);
        hipLaunchKernelGGL(gemm_f32, grid, dim3(256), 0, st, g);
        g.cfg = -1;
        log_launch(g, dtype);
    } else {
        if (int rc = prepare(g, dtype, false)) return rc;
        settle_rowsums(g);
        const int ap = settle_act(g, dtype);
        t_act_parts = g.c.act_mode == 2 ? ap : 0;
        if (dtype == G_F16) launch_t<half_t>(g, st);
        else launch_t<bf16_t>(g, st);
        log_launch(g, dtype);
    }
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return set_error(DM_ERR_DEVICE, "contraction launch: %s", hipGetErrorString(err));
    return 0;
}

int launch_gemm_pair(int dtype, const GemmArgs& x0, const GemmArgs& x1, hipStream_t st) {
    constexpr int64_t CUS = 256;
    t_rsum_parts = 0;
    if (dtype != G_F32 && x0.batch == 1 && x1.batch == 1 && x0.M > 0 && x0.N > 0 && x0.K > 0 && x1.M > 0 &&
        x1.N > 0 && x1.K > 0 && x0.a.kcontig == x1.a.kcontig && x0.b.kcontig == x1.b.kcontig) {
        GemmArgs g0 = x0, g1 = x1;
        if (int rc = prepare(g0, dtype, true)) return rc;
        if (int rc = prepare(g1, dtype, true)) return rc;
        // together the two fill the chip with one block per CU (fewer tiles
        // would leave CUs idle for the whole reduction, where separate
        // launches split it)
        const int64_t tiles = (int64_t)g0.tiles_m * g0.tiles_n + (int64_t)g1.tiles_m * g1.tiles_n;
        if (g0.cfg == 15 && g1.cfg == 15 && g0.splits == 1 && g1.splits == 1 && tiles >= CUS * 3 / 4 &&
            tiles <= CUS) {
            // the pair runs lean 128x128 tiles unsplit: row sums of either
            // operand A are produced (the first contraction's are reported)
            settle_rowsums(g1);
            settle_rowsums(g0);
            if (dtype == G_F16) launch_lean_pair<half_t, 128, 128, 2, 4, 64, 4>(g0, g1, st);
            else launch_lean_pair<bf16_t, 128, 128, 2, 4, 64, 4>(g0, g1, st);
            log_launch(g0, dtype);
            log_launch(g1, dtype);
            hipError_t err = hipGetLastError();
            if (err != hipSuccess) return set_error(DM_ERR_DEVICE, "contraction launch: %s", hipGetErrorString(err));
            return 0;
        }
    }
    if (int rc = launch_gemm(dtype, x0, st)) return rc;
    const int first_parts = t_rsum_parts;
    trace_next("2");
    const int rc = launch_gemm(dtype, x1, st);
    t_rsum_parts = first_parts;
    return rc;
}

}  // namespace dm
