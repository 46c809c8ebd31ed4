// Contraction kernels: every einsum of the layer (Fig. 1a and the
// Table 3 contraction rows, forward dX/dW split in backward) is one launch
// of a single MFMA GEMM whose operand and output addressing is general
// enough that no tensor is ever transposed or permuted in a separate pass.
//
// C[z][m][n] = alpha * sum_k A(z, m, k) * B(z, k, n)  (+ bias) (+ resid)
//
// Each operand is stored either contiguous along k ("k-contiguous": element
// (outer, k) at row(outer) + k) or contiguous along its outer index
// ("outer-contiguous": element (outer, k) at row(k) + outer).  The strided
// ("row") index goes through a mixed-radix map, which expresses plain
// strides, the paper's (p, h) <-> head-major (h, p) permutation, the split
// of a fused Q/K/V projection into per-head tensors, and a choice among up
// to three base pointers (the stacked [Wq Wk Wv] of algebraic fusion).
#pragma once

#include "common.hpp"

namespace dm {

// Mixed-radix index map: x = (d2 * r1 + d1) * r0 + d0, offset = d0*s0 + d1*s1
// + d2*s2 (elements).  r = 0 means the digit is unbounded.  When the map
// selects among several base pointers (nseg > 1) the top digit d2 picks the
// pointer and contributes no offset.
struct IdxMap {
    uint32_t r0, r1;
    uint32_t mul0, shr0, mul1, shr1;  // division by r0 / r1: q = (umulhi(x, mul) + x) >> shr
    int64_t s0, s1, s2;
};

__device__ __forceinline__ uint32_t fdiv(uint32_t x, uint32_t mul, uint32_t shr) {
    return (__umulhi(x, mul) + x) >> shr;
}

// offset and segment of index x
__device__ __forceinline__ int64_t map_off(const IdxMap& m, uint32_t x, int nseg, int* seg) {
    uint32_t d0 = x, d1 = 0, d2 = 0;
    if (m.r0) {
        uint32_t q = fdiv(x, m.mul0, m.shr0);
        d0 = x - q * m.r0;
        d1 = q;
        if (m.r1) { d2 = fdiv(q, m.mul1, m.shr1); d1 = q - d2 * m.r1; }
    }
    int64_t off = (int64_t)d0 * m.s0 + (int64_t)d1 * m.s1;
    if (nseg > 1) *seg = (int)d2; else off += (int64_t)d2 * m.s2;
    return off;
}

struct Operand {
    const void* ptr[3];
    int nseg;
    int kcontig;      // 1: rows indexed by the outer (m or n) index, contiguous along k
    IdxMap row;       // strided index -> offset
    IdxMap batch;     // z -> offset
};

struct Epilogue {
    void* ptr[3];
    int nseg;          // > 1: the segment digit of mmap (seg_on_m) or nmap picks the pointer
    int seg_on_m;
    IdxMap mmap, nmap, batch;
    int contig_n;      // 1: nmap has unit stride over aligned groups of 8; 0: mmap does
    float alpha;
    const void* bias[3];
    int bias_nseg;
    int bias_on_m;     // bias indexed by m instead of n
    IdxMap bias_map;
    const void* resid;  // optional, same addressing as C (single pointer)
    int out_f32;        // C (and resid) stored as float instead of the input dtype
    // optional: partial fp32 sums of A's rows over the contraction, as
    // rows of rsum (row stride rsum_ld >= M, at most rsum_cap rows); the sum
    // of partial rows 0 .. n-1 at column m is row m of A summed over k, with
    // n = gemm_rowsum_parts() after the launch (0: not produced, and rsum
    // untouched).  Only the lean 256x256 and 128x128 tiles, unsplit, with A
    // outer-contiguous produce them.
    float* rsum;
    int rsum_ld;
    int rsum_cap;
    // optional activation step in the epilogue (storage-type output, no
    // alpha scaling or bias; dropout element index m * ldc + n):
    // act_mode 1: also writes act_out = dropout(act(C + act_bias[n])) from
    // the stored (rounded) C;
    // act_mode 2: C is the gradient dA of the activation's output and is not
    // stored: C's pointer receives dH = dropout(dA) * act'(act_in + act_bias[n])
    // (dA rounded first, dH rounded as stored), and the partial column sums
    // of the stored dH go to rows of act_part (N floats each, at most
    // act_part_cap rows; gemm_act_parts() tells how many were written).
    // Only the staged epilogue of the lean kernels does this
    // (gemm_act_fusable tells beforehand).
    int act_mode;
    void* act_out;
    const void* act_in;
    const void* act_bias;
    int act;
    DropParams act_dp;
    float* act_part;
    int act_part_cap;
};

struct GemmArgs {
    int M, N, K, batch;
    Operand a, b;
    Epilogue c;
    int tiles_m, tiles_n;  // set by the launcher
    int splits;            // split-K factor; > 1 needs split_ws (0 or 1: none)
    float* split_ws;       // splits * batch * M * N floats of partial sums
    int64_t split_cap;     // floats available at split_ws
    int kper;              // k range per split (set by the launcher)
    int cfg;               // tile configuration index; < 0 lets the launcher choose
    // set by the launcher: outputs at coff(z) + m * ldc + n (contig_n) or
    // coff(z) + m + n * ldc, one pointer; bias_mode 0 none, 1 along the
    // contiguous output index (unit stride), 2 along the other index
    int affine, bias_mode;
    int64_t ldc;
    // set by the launcher: output maps affine over aligned blocks of 32
    // rows and columns (offsets then computed once per block)
    int blk32;
    // set by the launcher: the lean kernels may stage their output tile
    // through LDS and store 16-byte row pieces (bit 0: the output; bit 1:
    // split-k partials)
    int ep_stage;
};

// Number of Epilogue::rsum partial rows the last launch_gemm on this
// thread wrote (for launch_gemm_pair: its first contraction's), 0 if none.
int gemm_rowsum_parts();

// Whether launch_gemm would run this contraction with the staged epilogue
// that takes its Epilogue::act_mode step (otherwise the request is ignored
// and the caller applies the activation step itself).
bool gemm_act_fusable(int dtype, const GemmArgs& g);
// Partial column-sum rows the last launch_gemm on this thread wrote for
// act_mode 2 (0 if none).
int gemm_act_parts();

// Largest tile configuration index (contract's tile_cfg, plan entries).
constexpr int GEMM_MAX_CFG = 25;

// Scratch bytes for a split-K contraction.
inline size_t gemm_split_ws_bytes(int64_t M, int64_t N, int64_t batch, int splits) {
    return splits > 1 ? (size_t)splits * batch * M * N * sizeof(float) : 0;
}

// Host-side construction helpers.
IdxMap make_map(uint32_t r0, uint32_t r1, int64_t s0, int64_t s1, int64_t s2);
inline IdxMap linear_map(int64_t stride) { return make_map(0, 0, stride, 0, 0); }

enum GemmDtype { G_F32 = 0, G_F16 = 1, G_BF16 = 2 };

// Validates and launches one contraction; returns 0 on success, else a
// message is stored for dm_last_error and a nonzero code returned.
int launch_gemm(int dtype, const GemmArgs& args, hipStream_t stream);
// Two contractions in one launch when both take the lean 128x128 kernel
// unsplit with the same operand contiguity and their tiles together give
// between 3/4 of the CUs and all of them one block; otherwise launch_gemm on
// each, in order.
int launch_gemm_pair(int dtype, const GemmArgs& a, const GemmArgs& b, hipStream_t stream);

}  // namespace dm
