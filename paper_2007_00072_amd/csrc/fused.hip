// Memory-bound fused operators of the encoder layer (the paper's kernel
// list in Sec. "Fusion Implementation", Table 3 brackets), for gfx950.
//
// Row operators (LayerNorm and softmax, forward and backward) give each row
// to a group of LPR lanes of one wave64 (LPR = 64 for rows of 512..2048
// elements, fewer lanes for short rows so a wave holds several rows); each
// lane keeps NV 8-element vectors of its row in registers, so the
// reduce-then-apply structure of a statistical normalisation reads every
// input exactly once from HBM.  Reductions are xor-butterflies inside the
// lane group.  Dropout masks are regenerated with Philox from the logical
// element index, never loaded.  Column reductions (bias, LayerNorm scale
// and shift gradients) write per-block partial sums that a second small
// kernel adds in a fixed order, so results are deterministic.
#include <math.h>

#include "internal.hpp"

namespace dm {
namespace {

constexpr int NT = 256;  // threads per block: 4 wave64s

// ------------------------------------------------------ bias+dropout+residual+LayerNorm
template <typename T, int LPR, int NV>
__global__ __launch_bounds__(NT) void bdrln_fwd_k(int64_t rows, int cols, const T* __restrict__ x,
                                                  const T* __restrict__ bias, const T* __restrict__ resid,
                                                  const T* __restrict__ gamma, const T* __restrict__ beta,
                                                  float eps, DropParams dp, T* __restrict__ y,
                                                  T* __restrict__ xhat, float* __restrict__ rstd) {
    constexpr int RPW = 64 / LPR;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int gi = lane / LPR, gl = lane % LPR;
    const int64_t row = ((int64_t)blockIdx.x * 4 + wave) * RPW + gi;
    const bool active = row < rows;
    const int64_t base = row * cols;
    float v[NV][8];
    // v holds the row minus its first residual value r0: r - r0 is exact
    // for nearby values, so a row far from zero keeps its fp32 precision
    // (the sum a + r itself would lose it); the statistics and x_hat use
    // the shifted row throughout
    const float r0 = active ? to_f(resid[base]) : 0.f;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
        const int c = (gl + i * LPR) * 8;
        if (active && c < cols) {
            float a[8], b[8], r[8];
            V8<T>::load(x + base + c, a);
            V8<T>::load(bias + c, b);
            V8<T>::load(resid + base + c, r);
#pragma unroll
            for (int q = 0; q < 8; ++q) a[q] += b[q];
            dropout8(dp, (uint64_t)(base + c), a);
#pragma unroll
            for (int q = 0; q < 8; ++q) v[i][q] = (r[q] - r0) + a[q];
        } else {
#pragma unroll
            for (int q = 0; q < 8; ++q) v[i][q] = 0.f;
        }
    }
    const float inv = 1.0f / (float)cols;
    float ssum = 0.f;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
        const int c = (gl + i * LPR) * 8;
        if (active && c < cols) {
#pragma unroll
            for (int q = 0; q < 8; ++q) ssum += v[i][q];
        }
    }
    const float mean = group_sum<LPR>(ssum) * inv;  // of the shifted row
    float sq = 0.f;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
        const int c = (gl + i * LPR) * 8;
        if (active && c < cols) {
#pragma unroll
            for (int q = 0; q < 8; ++q) { float d = v[i][q] - mean; sq += d * d; }
        }
    }
    const float var = group_sum<LPR>(sq) * inv;
    const float rs = 1.0f / sqrtf(var + eps);
    if (!active) return;
    if (rstd && gl == 0) rstd[row] = rs;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
        const int c = (gl + i * LPR) * 8;
        if (c < cols) {
            float g[8], b[8], xh[8], o[8];
            V8<T>::load(gamma + c, g);
            V8<T>::load(beta + c, b);
#pragma unroll
            for (int q = 0; q < 8; ++q) { xh[q] = (v[i][q] - mean) * rs; o[q] = g[q] * xh[q] + b[q]; }
            V8<T>::store(y + base + c, o);
            if (xhat) V8<T>::store(xhat + base + c, xh);
        }
    }
}

// ------------------------------------------------------ scaled softmax + dropout
// Physical rows are [B][H][J]; the dropout logical index is (h, b, j, k).
// causal: keys k > j are masked (probability exactly zero).
template <typename T, int LPR, int NV>
__global__ __launch_bounds__(NT) void softmax_fwd_k(int64_t rows, int B, int H, int J, int K, float scale,
                                                    const T* __restrict__ beta, DropParams dp,
                                                    T* __restrict__ prob, T* __restrict__ alpha, int causal) {
    constexpr int RPW = 64 / LPR;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int gi = lane / LPR, gl = lane % LPR;
    const int64_t row = ((int64_t)blockIdx.x * 4 + wave) * RPW + gi;
    const bool active = row < rows;
    const int64_t base = row * K;
    const int kmax = causal ? (int)(row % J) : K - 1;  // last key the row sees
    float v[NV][8];
    float mx = -INFINITY;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
        const int c = (gl + i * LPR) * 8;
        if (active && c < K) {
            V8<T>::load(beta + base + c, v[i]);
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                v[i][q] = c + q <= kmax ? v[i][q] * scale : -INFINITY;
                mx = fmaxf(mx, v[i][q]);
            }
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
    if (!active) return;
    const float rinv = __builtin_amdgcn_rcpf(sum);
    const int j = (int)(row % J);
    const int64_t bh = row / J;
    const int h = (int)(bh % H), b = (int)(bh / H);
    const int64_t ebase = (((int64_t)h * B + b) * J + j) * (int64_t)K;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
        const int c = (gl + i * LPR) * 8;
        if (c < K) {
#pragma unroll
            for (int q = 0; q < 8; ++q) v[i][q] = to_f(from_f<T>(v[i][q] * rinv));  // P as stored
            V8<T>::store(prob + base + c, v[i]);
            dropout8(dp, (uint64_t)(ebase + c), v[i]);
            V8<T>::store(alpha + base + c, v[i]);
        }
    }
}

// ------------------------------------------------------ softmax + dropout backward
template <typename T, int LPR, int NV>
__global__ __launch_bounds__(NT) void softmax_bwd_k(int64_t rows, int B, int H, int J, int K, float scale,
                                                    const T* __restrict__ dalpha, const T* __restrict__ prob,
                                                    DropParams dp, T* __restrict__ dbeta) {
    constexpr int RPW = 64 / LPR;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int gi = lane / LPR, gl = lane % LPR;
    const int64_t row = ((int64_t)blockIdx.x * 4 + wave) * RPW + gi;
    const bool active = row < rows;
    const int64_t base = row * K;
    int64_t ebase = 0;
    if (active) {
        const int j = (int)(row % J);
        const int64_t bh = row / J;
        const int h = (int)(bh % H), b = (int)(bh / H);
        ebase = (((int64_t)h * B + b) * J + j) * (int64_t)K;
    }
    float dp_[NV][8], p[NV][8];
    float dot = 0.f;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
        const int c = (gl + i * LPR) * 8;
        if (active && c < K) {
            V8<T>::load(dalpha + base + c, dp_[i]);
            V8<T>::load(prob + base + c, p[i]);
            dropout8(dp, (uint64_t)(ebase + c), dp_[i]);
#pragma unroll
            for (int q = 0; q < 8; ++q) dot += dp_[i][q] * p[i][q];
        } else {
#pragma unroll
            for (int q = 0; q < 8; ++q) { dp_[i][q] = 0.f; p[i][q] = 0.f; }
        }
    }
    dot = group_sum<LPR>(dot);
    if (!active) return;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
        const int c = (gl + i * LPR) * 8;
        if (c < K) {
            float o[8];
#pragma unroll
            for (int q = 0; q < 8; ++q) o[q] = scale * p[i][q] * (dp_[i][q] - dot);
            V8<T>::store(dbeta + base + c, o);
        }
    }
}

// ------------------------------------------------------ alpha from the stored P
// alpha = dropout(P) re-formed from the saved probabilities (the forward
// forms it from the same rounded values and the same keep decisions, so the
// result is bit-identical); thread t handles 8 consecutive keys of one row.
template <typename T>
__global__ __launch_bounds__(256) void alpha_from_prob_k(int64_t n8, int B, int H, int J, int K,
                                                         const T* __restrict__ prob, DropParams dp,
                                                         T* __restrict__ alpha) {
    const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (t >= n8) return;
    const int64_t e = t * 8;
    const int64_t row = e / K;  // (b, h, j)
    const int c = (int)(e - row * K);
    const int j = (int)(row % J);
    const int64_t bh = row / J;
    const int h = (int)(bh % H), b = (int)(bh / H);
    float v[8];
    V8<T>::load(prob + e, v);
    dropout8(dp, (uint64_t)((((int64_t)h * B + b) * J + j) * (int64_t)K + c), v);
    V8<T>::store(alpha + e, v);
}

// ------------------------------------------------------ LayerNorm backward family
// Each block (8 waves) takes a contiguous range of rows; one lane group per
// row, so every wave has its own rows' loads in flight at once.  Column
// partial sums are kept per lane (a lane always owns the same columns),
// reduced over the wave's lane groups with shuffles and over the block's 8
// waves through LDS in a fixed order, and written as
// part[q][blockIdx.x][cols].
constexpr int NTL = 512;  // threads per LayerNorm-backward block

template <typename T, int LPR, int NV>
__global__ __launch_bounds__(NTL) void ln_bwd_k(LnBwdArgs a, int rows_per_block, int nblk) {
    constexpr int RPW = 64 / LPR;
    constexpr int GROUPS = (NTL / 64) * RPW;  // row slots per block iteration
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int gi = lane / LPR, gl = lane % LPR;
    const int cols = a.cols;
    const T* dya = reinterpret_cast<const T*>(a.dya);
    const T* dyb = reinterpret_cast<const T*>(a.dyb);
    const T* xhat = reinterpret_cast<const T*>(a.xhat);
    const T* gamma = reinterpret_cast<const T*>(a.gamma);
    const bool do_ds = a.ds || a.dsub;
    const bool do_part = a.part != nullptr;
    const int64_t r0 = (int64_t)blockIdx.x * rows_per_block;
    const int64_t r1 = min<int64_t>(a.rows, r0 + rows_per_block);

    float g[NV][8];
    float p_dyx[NV][8], p_dy[NV][8], p_dsub[NV][8];
#pragma unroll
    for (int i = 0; i < NV; ++i) {
        const int c = (gl + i * LPR) * 8;
        if (do_ds && c < cols) V8<T>::load(gamma + c, g[i]);
#pragma unroll
        for (int q = 0; q < 8; ++q) { p_dyx[i][q] = 0.f; p_dy[i][q] = 0.f; p_dsub[i][q] = 0.f; }
    }

    // UR rows per lane group are in flight: all their loads are issued
    // before the first row's reductions.
    constexpr int UR = NV <= 2 ? 2 : 1;
    for (int64_t rb = r0; rb < r1; rb += GROUPS * UR) {
        float dy[UR][NV][8], xh[UR][NV][8], rsv[UR];
#pragma unroll
        for (int u = 0; u < UR; ++u) {
            const int64_t row = rb + u * GROUPS + wave * RPW + gi;
            const bool active = row < r1;
            const int64_t base = row * cols;
            // the row's 1/std is loaded with its other inputs, not after the
            // reductions (a load issued there costs a full memory latency)
            rsv[u] = do_ds && active ? a.rstd[row] : 0.f;
#pragma unroll
            for (int i = 0; i < NV; ++i) {
                const int c = (gl + i * LPR) * 8;
                if (active && c < cols) {
                    V8<T>::load(dya + base + c, dy[u][i]);
                    V8<T>::load(xhat + base + c, xh[u][i]);
                    if (dyb) {
                        float t[8];
                        V8<T>::load(dyb + base + c, t);
#pragma unroll
                        for (int q = 0; q < 8; ++q) dy[u][i][q] += t[q];
                    }
                } else {
#pragma unroll
                    for (int q = 0; q < 8; ++q) { dy[u][i][q] = 0.f; xh[u][i][q] = 0.f; }
                }
            }
        }
#pragma unroll
        for (int u = 0; u < UR; ++u) {
            const int64_t row = rb + u * GROUPS + wave * RPW + gi;
            const bool active = row < r1;
            const int64_t base = row * cols;
            float s1 = 0.f, s2 = 0.f;
#pragma unroll
            for (int i = 0; i < NV; ++i) {
                const int c = (gl + i * LPR) * 8;
                if (active && c < cols) {
                    if (a.dysum) V8<T>::store(reinterpret_cast<T*>(a.dysum) + base + c, dy[u][i]);
#pragma unroll
                    for (int q = 0; q < 8; ++q) {
                        if (do_part) { p_dyx[i][q] += dy[u][i][q] * xh[u][i][q]; p_dy[i][q] += dy[u][i][q]; }
                        if (do_ds) { float gy = dy[u][i][q] * g[i][q]; s1 += gy; s2 += gy * xh[u][i][q]; }
                    }
                }
            }
            if (do_ds) {
                const float inv = 1.0f / (float)cols;
                const float m1 = group_sum<LPR>(s1) * inv;
                const float m2 = group_sum<LPR>(s2) * inv;
                if (active) {
                    const float rs = rsv[u];
#pragma unroll
                    for (int i = 0; i < NV; ++i) {
                        const int c = (gl + i * LPR) * 8;
                        if (c < cols) {
                            float o[8];
#pragma unroll
                            for (int q = 0; q < 8; ++q) o[q] = rs * (dy[u][i][q] * g[i][q] - m1 - xh[u][i][q] * m2);
                            if (a.ds) V8<T>::store(reinterpret_cast<T*>(a.ds) + base + c, o);
                            if (a.dsub) {
                                dropout8(a.dp, (uint64_t)(base + c), o);
                                V8<T>::store(reinterpret_cast<T*>(a.dsub) + base + c, o);
                                if (do_part && a.want_dsub_sum) {
                                    // sum the stored (rounded) values that later consumers see
#pragma unroll
                                    for (int q = 0; q < 8; ++q) p_dsub[i][q] += to_f(from_f<T>(o[q]));
                                }
                            }
                        }
                    }
                }
            }
        }
    }
    if (!do_part) return;

    // reduce partials over the RPW lane groups of the wave
    __shared__ float red[NTL / 64][2048];
    const int nq = a.want_dsub_sum ? 3 : 2;
    for (int qn = 0; qn < nq; ++qn) {
        float(*pp)[8] = qn == 0 ? p_dyx : (qn == 1 ? p_dy : p_dsub);
#pragma unroll
        for (int i = 0; i < NV; ++i)
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                float t = pp[i][q];
#pragma unroll
                for (int o = LPR; o < 64; o <<= 1) t += __shfl_xor(t, o, 64);
                pp[i][q] = t;
            }
        __syncthreads();
        if (gi == 0) {
#pragma unroll
            for (int i = 0; i < NV; ++i) {
                const int c = (gl + i * LPR) * 8;
                if (c < cols) {
#pragma unroll
                    for (int q = 0; q < 8; ++q) red[wave][c + q] = pp[i][q];
                }
            }
        }
        __syncthreads();
        float* out = a.part + ((int64_t)qn * nblk + blockIdx.x) * cols;
        for (int c = threadIdx.x; c < cols; c += NTL)
            out[c] = ((red[0][c] + red[1][c]) + (red[2][c] + red[3][c])) +
                     ((red[4][c] + red[5][c]) + (red[6][c] + red[7][c]));
    }
}

// ------------------------------------------------------ activation backward + bias grad
// Block (x, y) takes the rows of row block x and the column chunk y of
// NT*8 columns: each thread owns one 8-column vector and walks its rows
// four at a time (all loads of the four rows issued before any use).
constexpr int RU = 4;

template <typename T>
__global__ __launch_bounds__(NT) void act_bwd_k(int64_t rows, int F, const T* __restrict__ da,
                                                const T* __restrict__ h, const T* __restrict__ b1, int act,
                                                DropParams dp, T* __restrict__ dh, float* __restrict__ part,
                                                int rows_per_block) {
    const int v = blockIdx.y * NT + threadIdx.x;
    if (v >= F / 8) return;
    const int64_t r0 = (int64_t)blockIdx.x * rows_per_block;
    const int64_t r1 = min<int64_t>(rows, r0 + rows_per_block);
    float bb[8], acc[8];
    V8<T>::load(b1 + v * 8, bb);
#pragma unroll
    for (int q = 0; q < 8; ++q) acc[q] = 0.f;
    for (int64_t r = r0; r < r1; r += RU) {
        float g[RU][8], u[RU][8];
#pragma unroll
        for (int j = 0; j < RU; ++j)
            if (r + j < r1) {
                V8<T>::load(da + (r + j) * F + v * 8, g[j]);
                V8<T>::load(h + (r + j) * F + v * 8, u[j]);
            }
#pragma unroll
        for (int j = 0; j < RU; ++j)
            if (r + j < r1) {
                const int64_t off = (r + j) * F + v * 8;
                dropout8(dp, (uint64_t)off, g[j]);
#pragma unroll
                for (int q = 0; q < 8; ++q) g[j][q] *= act_grad(u[j][q] + bb[q], act);
                V8<T>::store(dh + off, g[j]);
                // sum the stored (rounded) values that consumers of dh read
#pragma unroll
                for (int q = 0; q < 8; ++q) acc[q] += to_f(from_f<T>(g[j][q]));
            }
    }
    V8<float>::store(part + (int64_t)blockIdx.x * F + v * 8, acc);
}

// The same, also writing dh transposed (dht[f][row], the layout in which
// the Linear-1 weight gradient reads it contiguous along the tokens): rows
// go in groups of 8, so each lane writes every one of its 8 columns as one
// 16-byte piece of 8 consecutive rows.  Blocks are numbered so that each
// XCD takes one contiguous eighth of the rows: the pieces of one 128-byte
// line of dht (64 rows, 8 row blocks) are then written through one L2,
// which merges them before they reach HBM.  Needs rows and
// rows_per_block multiples of 8.
template <typename T>
__global__ __launch_bounds__(NT) void act_bwd_t_k(int64_t rows, int F, const T* __restrict__ da,
                                                  const T* __restrict__ h, const T* __restrict__ b1, int act,
                                                  DropParams dp, T* __restrict__ dh, T* __restrict__ dht,
                                                  float* __restrict__ part, int rows_per_block, int nrb) {
    const int lid = (int)blockIdx.x, total = (int)gridDim.x;
    int rb, cb;
    if ((nrb & 7) == 0 && (total & 7) == 0) {
        const int per = nrb >> 3, i = lid >> 3;
        cb = i / per;
        rb = (lid & 7) * per + (i - cb * per);
    } else {
        cb = lid / nrb;
        rb = lid - cb * nrb;
    }
    const int v = cb * NT + threadIdx.x;
    if (v >= F / 8) return;
    const int64_t r0 = (int64_t)rb * rows_per_block;
    const int64_t r1 = min<int64_t>(rows, r0 + rows_per_block);
    float bb[8], acc[8];
    V8<T>::load(b1 + v * 8, bb);
#pragma unroll
    for (int q = 0; q < 8; ++q) acc[q] = 0.f;
    for (int64_t r = r0; r < r1; r += 8) {
        float g[8][8], u[8][8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            V8<T>::load(da + (r + j) * F + v * 8, g[j]);
            V8<T>::load(h + (r + j) * F + v * 8, u[j]);
        }
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int64_t off = (r + j) * F + v * 8;
            dropout8(dp, (uint64_t)off, g[j]);
#pragma unroll
            for (int q = 0; q < 8; ++q) g[j][q] = to_f(from_f<T>(g[j][q] * act_grad(u[j][q] + bb[q], act)));
            V8<T>::store(dh + off, g[j]);
#pragma unroll
            for (int q = 0; q < 8; ++q) acc[q] += g[j][q];
        }
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            float col[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) col[j] = g[j][q];
            V8<T>::store(dht + (int64_t)(v * 8 + q) * rows + r, col);
        }
    }
    V8<float>::store(part + (int64_t)rb * F + v * 8, acc);
}

template <typename T>
__global__ __launch_bounds__(NT) void colsum_partial_k(int64_t rows, int cols, const T* __restrict__ x,
                                                       float* __restrict__ part, int rows_per_block) {
    const int v = blockIdx.y * NT + threadIdx.x;
    if (v >= cols / 8) return;
    const int64_t r0 = (int64_t)blockIdx.x * rows_per_block;
    const int64_t r1 = min<int64_t>(rows, r0 + rows_per_block);
    float acc[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) acc[q] = 0.f;
    for (int64_t r = r0; r < r1; r += RU) {
        float t[RU][8];
#pragma unroll
        for (int j = 0; j < RU; ++j)
            if (r + j < r1) V8<T>::load(x + (r + j) * cols + v * 8, t[j]);
#pragma unroll
        for (int j = 0; j < RU; ++j)
            if (r + j < r1) {
#pragma unroll
                for (int q = 0; q < 8; ++q) acc[q] += t[j][q];
            }
    }
    V8<float>::store(part + (int64_t)blockIdx.x * cols + v * 8, acc);
}

// out[c] = sum over the nblk partial rows in a fixed order.  A launch runs
// a list of jobs (partial sets of several operators, finished together);
// each block finds its job from the jobs' first-block table, then covers
// columns 32x .. 32x+31 of one partial set (a whole 128-byte line of every
// partial row) as 8 four-column groups x 64 row phases; each phase sums
// rows ph, ph+64, ... with eight loads in flight (one memory round trip
// for 512 partial rows).  The phase sums are added as a fixed tree: the 8
// phases of a wave by butterfly shuffles, then the 8 waves' sums in wave
// order.  Set y of a job is part + y*nblk*cols -> out[y].  With qkv_H > 0
// the columns are (s, h, p) of a fused projection and land in
// out[s][p * qkv_H + h] (single partial set).
constexpr int FIN_COLS = 32;
constexpr int FIN_NT = 512;

__global__ __launch_bounds__(FIN_NT) void colsum_finish_k(FinishJobs fj) {
    constexpr int CG = FIN_COLS / 4, NPH = FIN_NT / CG, NWV = FIN_NT / 64;  // column groups, row phases, waves
    __shared__ floatx4 red[NWV][CG];
    int jb = 0;
#pragma unroll
    for (int i = 1; i < MAX_FINISH_JOBS; ++i)
        if (i < fj.n && (int)blockIdx.x >= fj.first[i]) jb = i;
    const FinishJob& job = fj.job[jb];
    const int cols = job.cols, nblk = job.nblk;
    const int local = (int)blockIdx.x - fj.first[jb];
    const int ncb = (cols + FIN_COLS - 1) / FIN_COLS;
    const int set = local / ncb, cbk = local - set * ncb;
    const int cg = threadIdx.x % CG, ph = threadIdx.x / CG, wave = threadIdx.x / 64;
    const int c = cbk * FIN_COLS + cg * 4;
    const float* base = job.part + (int64_t)set * nblk * cols;
    constexpr int U = 8;
    floatx4 s[U];
#pragma unroll
    for (int u = 0; u < U; ++u) s[u] = floatx4{0.f, 0.f, 0.f, 0.f};
    if (c < cols) {
        for (int b = ph; b < nblk; b += U * NPH) {
            floatx4 t[U];
#pragma unroll
            for (int u = 0; u < U; ++u)
                t[u] = b + NPH * u < nblk ? *reinterpret_cast<const floatx4*>(base + (int64_t)(b + NPH * u) * cols + c)
                                          : floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int u = 0; u < U; ++u) s[u] += t[u];
        }
    }
    floatx4 t = ((s[0] + s[1]) + (s[2] + s[3])) + ((s[4] + s[5]) + (s[6] + s[7]));
    // the wave's 8 phases of this column group (lanes cg, cg + 8, ..., cg + 56)
#pragma unroll
    for (int d = CG; d < 64; d <<= 1)
#pragma unroll
        for (int q = 0; q < 4; ++q) t[q] += __shfl_xor(t[q], d, 64);
    if ((threadIdx.x & 63) < CG) red[wave][cg] = t;
    __syncthreads();
    if (threadIdx.x < CG && c < cols) {
        floatx4 tot = red[0][cg];
#pragma unroll
        for (int w = 1; w < NWV; ++w) tot += red[w][cg];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int cc = c + q;
            if (job.qkv_H > 0) {
                // column (s, h, p) of a fused projection -> bias gradient b_s[p][h]
                const int I = job.qkv_H * job.qkv_P;
                const int sg = cc / I, hp = cc - sg * I, hh = hp / job.qkv_P, pp = hp - hh * job.qkv_P;
                job.out[sg][pp * job.qkv_H + hh] = tot[q];
            } else {
                job.out[set][cc] = tot[q];
            }
        }
    }
}

// ------------------------------------------------------ element-wise
template <typename T>
__global__ __launch_bounds__(NT) void bias_act_fwd_k(int64_t nvec, int cols, const T* __restrict__ x,
                                                     const T* __restrict__ bias, int act, DropParams dp,
                                                     T* __restrict__ y) {
    const int cv = cols / 8;
    for (int64_t v = (int64_t)blockIdx.x * NT + threadIdx.x; v < nvec; v += (int64_t)gridDim.x * NT) {
        const int64_t r = v / cv;
        const int c = (int)(v - r * cv) * 8;
        float a[8], b[8];
        V8<T>::load(x + r * cols + c, a);
        V8<T>::load(bias + c, b);
#pragma unroll
        for (int q = 0; q < 8; ++q) a[q] = act_fwd(a[q] + b[q], act);
        dropout8(dp, (uint64_t)(r * cols + c), a);
        V8<T>::store(y + r * cols + c, a);
    }
}

template <typename T>
__global__ __launch_bounds__(NT) void attn_input_bias_k(int64_t nvec, int H, int P, const T* __restrict__ x,
                                                        const T* __restrict__ bq, const T* __restrict__ bk,
                                                        const T* __restrict__ bv, T* __restrict__ y) {
    const int I = H * P, rowv = 3 * I / 8;
    for (int64_t v = (int64_t)blockIdx.x * NT + threadIdx.x; v < nvec; v += (int64_t)gridDim.x * NT) {
        const int64_t r = v / rowv;
        const int c = (int)(v - r * rowv) * 8;
        const int s = c / I, hp = c - s * I, hh = hp / P, p0 = hp - hh * P;
        const T* b = s == 0 ? bq : (s == 1 ? bk : bv);
        float a[8];
        V8<T>::load(x + r * 3 * I + c, a);
#pragma unroll
        for (int q = 0; q < 8; ++q) a[q] += to_f(b[(p0 + q) * H + hh]);
        V8<T>::store(y + r * 3 * I + c, a);
    }
}

template <typename T>
__global__ __launch_bounds__(NT) void add_k(int64_t nvec, const T* __restrict__ a, const T* __restrict__ b,
                                            T* __restrict__ out) {
    for (int64_t v = (int64_t)blockIdx.x * NT + threadIdx.x; v < nvec; v += (int64_t)gridDim.x * NT) {
        float x[8], y[8];
        V8<T>::load(a + v * 8, x);
        V8<T>::load(b + v * 8, y);
#pragma unroll
        for (int q = 0; q < 8; ++q) x[q] += y[q];
        V8<T>::store(out + v * 8, x);
    }
}

// one wave per row: out[r] = sum over the row (fixed lane order, then butterfly)
template <typename T>
__global__ __launch_bounds__(NT) void rowsum_k(int64_t rows, int len, const T* __restrict__ x,
                                               float* __restrict__ out) {
    const int lane = threadIdx.x & 63;
    const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (r >= rows) return;
    float s = 0.f;
    for (int c = lane * 8; c < len; c += 512) {
        float v[8];
        V8<T>::load(x + r * len + c, v);
#pragma unroll
        for (int q = 0; q < 8; ++q) s += v[q];
    }
    s = group_sum<64>(s);
    if (lane == 0) out[r] = s;
}

__global__ __launch_bounds__(NT) void dropout_mask_k(DropParams dp, uint64_t offset, uint64_t nvec,
                                                     uint8_t* __restrict__ out) {
    for (uint64_t v = (uint64_t)blockIdx.x * NT + threadIdx.x; v < nvec; v += (uint64_t)gridDim.x * NT) {
        uint8_t k[8];
        keep8(dp, offset + v * 8, k);
        u32x2 w;
        w[0] = k[0] | (k[1] << 8) | (k[2] << 16) | ((uint32_t)k[3] << 24);
        w[1] = k[4] | (k[5] << 8) | (k[6] << 16) | ((uint32_t)k[7] << 24);
        *reinterpret_cast<u32x2*>(out + v * 8) = w;
    }
}

int grid_for(int64_t nvec) {
    int64_t g = (nvec + NT - 1) / NT;
    return (int)(g < 8192 ? (g < 1 ? 1 : g) : 8192);
}

// Row-kernel dispatch on the row length: (lanes per row, vectors per lane).
#define DM_ROW_CASES(LAUNCH)                                                   \
    if (len <= 32) { LAUNCH(4, 1); }                                           \
    else if (len <= 64) { LAUNCH(8, 1); }                                      \
    else if (len <= 128) { LAUNCH(16, 1); }                                    \
    else if (len <= 256) { LAUNCH(32, 1); }                                    \
    else if (len <= 512) { LAUNCH(64, 1); }                                    \
    else if (len <= 1024) { LAUNCH(64, 2); }                                   \
    else if (len <= 2048) { LAUNCH(64, 4); }                                   \
    else { LAUNCH(64, 8); }

// Lanes per row chosen by a configuration plan (the reduction width of a
// row operator): 32 or 16 lanes per row for rows of 257..1024 elements, each
// lane holding proportionally more vectors; anything else takes the table
// above.
#define DM_ROW_CASES_LANES(lanes, LAUNCH)                                          \
    if ((lanes) == 32 && len > 256 && len <= 1024) {                               \
        if (len <= 512) { LAUNCH(32, 2); }                                         \
        else if (len <= 768) { LAUNCH(32, 3); }                                    \
        else { LAUNCH(32, 4); }                                                    \
    } else if ((lanes) == 16 && len > 256 && len <= 1024) {                        \
        if (len <= 512) { LAUNCH(16, 4); }                                         \
        else if (len <= 768) { LAUNCH(16, 6); }                                    \
        else { LAUNCH(16, 8); }                                                    \
    } else { DM_ROW_CASES(LAUNCH) }

template <typename T>
void bdrln_t(int64_t rows, int len, const void* x, const void* bias, const void* resid, const void* gamma,
             const void* beta, float eps, const DropParams& dp, void* y, void* xhat, float* rstd,
             int lanes, hipStream_t st) {
#define L(LPR, NV)                                                                              \
    {                                                                                           \
        int64_t rpb = 4 * (64 / LPR);                                                           \
        hipLaunchKernelGGL((bdrln_fwd_k<T, LPR, NV>), dim3((rows + rpb - 1) / rpb), dim3(NT), 0, \
                           st, rows, len, (const T*)x, (const T*)bias, (const T*)resid,         \
                           (const T*)gamma, (const T*)beta, eps, dp, (T*)y, (T*)xhat, rstd);    \
    }
    DM_ROW_CASES_LANES(lanes, L)
#undef L
}

template <typename T>
void softmax_t(int B, int H, int J, int len, float scale, const void* beta, const DropParams& dp,
               void* prob, void* alpha, int causal, hipStream_t st) {
    int64_t rows = (int64_t)B * H * J;
#define L(LPR, NV)                                                                                \
    {                                                                                             \
        int64_t rpb = 4 * (64 / LPR);                                                             \
        hipLaunchKernelGGL((softmax_fwd_k<T, LPR, NV>), dim3((rows + rpb - 1) / rpb), dim3(NT), 0, \
                           st, rows, B, H, J, len, scale, (const T*)beta, dp, (T*)prob, (T*)alpha, causal); \
    }
    DM_ROW_CASES(L)
#undef L
}

template <typename T>
void softmax_bwd_t(int B, int H, int J, int len, float scale, const void* dalpha, const void* prob,
                   const DropParams& dp, void* dbeta, hipStream_t st) {
    int64_t rows = (int64_t)B * H * J;
#define L(LPR, NV)                                                                                \
    {                                                                                             \
        int64_t rpb = 4 * (64 / LPR);                                                             \
        hipLaunchKernelGGL((softmax_bwd_k<T, LPR, NV>), dim3((rows + rpb - 1) / rpb), dim3(NT), 0, \
                           st, rows, B, H, J, len, scale, (const T*)dalpha, (const T*)prob, dp,   \
                           (T*)dbeta);                                                            \
    }
    DM_ROW_CASES(L)
#undef L
}

// Column-split form for rows of 320 .. 1024 elements (multiples of 64):
// the block's 8 waves own 8 column slices of 16-row tiles, a lane group of
// LG lanes (a power of two covering the slice's cols/64 vectors) takes one
// row of its slice, and a wave covers 64/LG rows per pass.  The row
// statistics need the whole row: each lane group reduces its slice with
// DPP steps and the 8 slice sums meet in LDS, added in slice order (the
// tiles alternate between two LDS halves, so one barrier per tile
// suffices).  Column partial sums never leave their wave: a lane keeps
// its 8 columns' sums over all the rows it sees, the wave's lane groups
// are added with shuffles at the end, and lane group 0 writes
// part[q][blockIdx.x][columns].  Blocks stride over the tiles, so the
// partial count is ln_bwd_blocks(rows, cols).  The blocks of each XCD take
// a contiguous run of tiles, so the 32-byte pieces of one 128-byte line of
// the transposed copy meet in one L2.
constexpr int LN_TILE = 16;

template <typename T, int LG>
__global__ __launch_bounds__(NTL) void ln_bwd_cs_k(LnBwdArgs a, int nblk) {
    constexpr int NW = NTL / 64;       // column slices
    constexpr int RPP = 64 / LG;       // rows per pass of one wave
    constexpr int NP = LN_TILE / RPP;  // passes per tile
    static_assert(NP >= 1 && NP * RPP == LN_TILE, "tile rows");
    __shared__ float rowred[2][LN_TILE][NW][2];
    // transposed copy of the tile's dsub (16-bit types): column c's LN_TILE
    // rows at tb[c * LN_TILE ..], written out as 32-byte row pieces of
    // dsub_t[c][t0 ..]
    __shared__ __attribute__((aligned(16))) uint16_t tb[1024 * LN_TILE];
    static_assert(LN_TILE == 16, "a tile column is written as two 16-byte pieces");
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int gi = lane / LG, v = lane % LG;
    const int cols = a.cols, vpr = cols / (8 * NW);
    const bool vact = v < vpr;
    const int c = (wave * vpr + (vact ? v : 0)) * 8;  // this lane's 8 columns (idle lanes alias the slice's first)
    const T* dya = reinterpret_cast<const T*>(a.dya);
    const T* dyb = reinterpret_cast<const T*>(a.dyb);
    const T* xhat = reinterpret_cast<const T*>(a.xhat);
    const bool do_ds = a.ds || a.dsub;
    const bool do_part = a.part != nullptr;
    const float inv = 1.0f / (float)cols;

    float g[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) g[q] = 0.f;
    if (do_ds) V8<T>::load(reinterpret_cast<const T*>(a.gamma) + c, g);
    float p_dyx[8], p_dy[8], p_dsub[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) { p_dyx[q] = 0.f; p_dy[q] = 0.f; p_dsub[q] = 0.f; }

    int buf = 0;
    // block -> tile: XCD x (blocks x, x + 8, ...) takes tiles
    // x * nblk / 8 .. of every round of nblk tiles
    const int b = (int)blockIdx.x;
    const int tb0 = (nblk & 7) == 0 ? (b & 7) * (nblk >> 3) + (b >> 3) : b;
    for (int64_t t0 = (int64_t)tb0 * LN_TILE; t0 < a.rows; t0 += (int64_t)nblk * LN_TILE, buf ^= 1) {
        // every load of the tile is issued before any arithmetic (rows past
        // the end re-read the tile's first row; their results are dropped)
        u32x4 ldy[NP], lxh[NP], ldb[NP];
        float rs[NP];
#pragma unroll
        for (int p = 0; p < NP; ++p) {
            const int64_t row = t0 + p * RPP + gi;
            const int64_t rr = row < a.rows ? row : t0;
            ldy[p] = *reinterpret_cast<const u32x4*>(dya + rr * cols + c);
            lxh[p] = *reinterpret_cast<const u32x4*>(xhat + rr * cols + c);
            if (dyb) ldb[p] = *reinterpret_cast<const u32x4*>(dyb + rr * cols + c);
            rs[p] = do_ds ? a.rstd[rr] : 0.f;
        }
        float dy[NP][8], xh[NP][8];
#pragma unroll
        for (int p = 0; p < NP; ++p) {
            V8<T>::unpack(ldy[p], dy[p]);
            V8<T>::unpack(lxh[p], xh[p]);
            if (dyb) {
                float t[8];
                V8<T>::unpack(ldb[p], t);
#pragma unroll
                for (int q = 0; q < 8; ++q) dy[p][q] += t[q];
            }
        }
        if (do_ds) {
#pragma unroll
            for (int p = 0; p < NP; ++p) {
                float s1 = 0.f, s2 = 0.f;
                if (vact) {
#pragma unroll
                    for (int q = 0; q < 8; ++q) { const float gy = dy[p][q] * g[q]; s1 += gy; s2 += gy * xh[p][q]; }
                }
                s1 = group_sum<LG>(s1);
                s2 = group_sum<LG>(s2);
                if (v == 0) {
                    rowred[buf][p * RPP + gi][wave][0] = s1;
                    rowred[buf][p * RPP + gi][wave][1] = s2;
                }
            }
            __syncthreads();
        }
#pragma unroll
        for (int p = 0; p < NP; ++p) {
            const int64_t row = t0 + p * RPP + gi;
            const bool act = row < a.rows && vact;
            const int64_t off = row * cols + c;
            if (act && a.dysum) V8<T>::store(reinterpret_cast<T*>(a.dysum) + off, dy[p]);
            if (act && do_part) {
#pragma unroll
                for (int q = 0; q < 8; ++q) { p_dyx[q] += dy[p][q] * xh[p][q]; p_dy[q] += dy[p][q]; }
            }
            if (!do_ds) continue;
            float m1 = 0.f, m2 = 0.f;
#pragma unroll
            for (int w = 0; w < NW; ++w) { m1 += rowred[buf][p * RPP + gi][w][0]; m2 += rowred[buf][p * RPP + gi][w][1]; }
            m1 *= inv;
            m2 *= inv;
            if (!act) continue;
            float o[8];
#pragma unroll
            for (int q = 0; q < 8; ++q) o[q] = rs[p] * (dy[p][q] * g[q] - m1 - xh[p][q] * m2);
            if (a.ds) V8<T>::store(reinterpret_cast<T*>(a.ds) + off, o);
            if (a.dsub) {
                dropout8(a.dp, (uint64_t)off, o);
                V8<T>::store(reinterpret_cast<T*>(a.dsub) + off, o);
                if constexpr (sizeof(T) == 2) {
                    if (a.dsub_t) {
                        const int r = p * RPP + gi;  // row within the tile
#pragma unroll
                        for (int q = 0; q < 8; ++q) tb[(c + q) * LN_TILE + r] = __builtin_bit_cast(uint16_t, from_f<T>(o[q]));
                    }
                }
                if (do_part && a.want_dsub_sum) {
                    // sum the stored (rounded) values that later consumers see
#pragma unroll
                    for (int q = 0; q < 8; ++q) p_dsub[q] += to_f(from_f<T>(o[q]));
                }
            }
        }
        if constexpr (sizeof(T) == 2) {
            if (a.dsub_t && a.dsub && do_ds) {
                // the tile's transposed dsub: each column's (up to) LN_TILE
                // rows as one 32-byte piece of dsub_t[c][t0 ..] (rows and t0
                // multiples of 8 keep the pieces 16-byte aligned); the last,
                // partial tile element by element
                __syncthreads();
                const int nr = (int)min<int64_t>(LN_TILE, a.rows - t0);
                uint16_t* dtr = reinterpret_cast<uint16_t*>(a.dsub_t);
                if (nr == LN_TILE && (a.rows & 7) == 0) {
                    // lanes 2i and 2i+1 store the two halves of one column's
                    // 32 bytes, so each store instruction writes 32-byte runs
                    for (int idx = (int)threadIdx.x; idx < 2 * cols; idx += NTL) {
                        const int col = idx >> 1, h8 = (idx & 1) * 8;
                        *reinterpret_cast<u32x4*>(dtr + (int64_t)col * a.rows + t0 + h8) =
                            *reinterpret_cast<const u32x4*>(tb + col * LN_TILE + h8);
                    }
                } else {
                    for (int col = (int)threadIdx.x; col < cols; col += NTL) {
                        const uint16_t* src = tb + col * LN_TILE;
                        uint16_t* dst = dtr + (int64_t)col * a.rows + t0;
                        for (int r = 0; r < nr; ++r) dst[r] = src[r];
                    }
                }
                __syncthreads();  // the next tile rewrites tb
            }
        }
    }
    if (!do_part) return;
    const int nq = a.want_dsub_sum ? 3 : 2;
    for (int qn = 0; qn < nq; ++qn) {
        float* pp = qn == 0 ? p_dyx : (qn == 1 ? p_dy : p_dsub);
        float o[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            float t = pp[q];
#pragma unroll
            for (int d = LG; d < 64; d <<= 1) t += __shfl_xor(t, d, 64);
            o[q] = t;
        }
        if (gi == 0 && vact) V8<float>::store(a.part + ((int64_t)qn * nblk + blockIdx.x) * cols + c, o);
    }
}

template <typename T>
void ln_bwd_t(const LnBwdArgs& a, hipStream_t st) {
    const int nblk = ln_bwd_blocks(a.rows, a.cols, a.dtype, a.form);
    if constexpr (sizeof(T) == 2) {
        if (ln_bwd_uses_split(a.cols, a.dtype, a.form)) {
            if (a.cols / 64 <= 8) hipLaunchKernelGGL((ln_bwd_cs_k<T, 8>), dim3(nblk), dim3(NTL), 0, st, a, nblk);
            else hipLaunchKernelGGL((ln_bwd_cs_k<T, 16>), dim3(nblk), dim3(NTL), 0, st, a, nblk);
            return;
        }
    }
    const int len = a.cols;
    const int rpb = (int)((a.rows + nblk - 1) / nblk);
#define L(LPR, NV) \
    { hipLaunchKernelGGL((ln_bwd_k<T, LPR, NV>), dim3(nblk), dim3(NTL), 0, st, a, rpb, nblk); }
    DM_ROW_CASES_LANES(a.lanes, L)
#undef L
}

}  // namespace

int act_bwd_blocks(int64_t rows, bool transposed) {
    const int nblk = colsum_blocks(rows);
    if (!transposed) return nblk;
    const int rpb = (int)((rows + nblk - 1) / nblk + 7) / 8 * 8;
    return (int)((rows + rpb - 1) / rpb);
}

int colsum_blocks(int64_t rows) {
    int64_t b = (rows + 7) / 8;
    if (b > 512) b = 512;
    return (int)(b < 1 ? 1 : b);
}

int ln_bwd_blocks(int64_t rows, int cols, int dtype, int form) {
    if (!ln_bwd_uses_split(cols, dtype, form)) return colsum_blocks(rows);
    int64_t b = (rows + LN_TILE - 1) / LN_TILE;
    if (b > 512) b = 512;
    return (int)(b < 1 ? 1 : b);
}

#define DM_DTYPE_SWITCH(dtype, ...)                                \
    do {                                                           \
        if ((dtype) == DM_F32) { typedef float T; __VA_ARGS__; }   \
        else if ((dtype) == DM_F16) { typedef half_t T; __VA_ARGS__; } \
        else { typedef bf16_t T; __VA_ARGS__; }                    \
    } while (0)

void run_bdrln_fwd(int dtype, int64_t rows, int cols, const void* x, const void* bias, const void* resid,
                   const void* gamma, const void* beta, float eps, const DropParams& dp, void* y, void* xhat,
                   float* rstd, hipStream_t st, int lanes) {
    DM_DTYPE_SWITCH(dtype, bdrln_t<T>(rows, cols, x, bias, resid, gamma, beta, eps, dp, y, xhat, rstd, lanes, st));
}

void run_softmax_fwd(int dtype, int B, int H, int J, int K, float scale, const void* beta, const DropParams& dp,
                     void* prob, void* alpha, hipStream_t st, int causal) {
    DM_DTYPE_SWITCH(dtype, softmax_t<T>(B, H, J, K, scale, beta, dp, prob, alpha, causal, st));
}

void run_softmax_bwd(int dtype, int B, int H, int J, int K, float scale, const void* dalpha, const void* prob,
                     const DropParams& dp, void* dbeta, hipStream_t st) {
    DM_DTYPE_SWITCH(dtype, softmax_bwd_t<T>(B, H, J, K, scale, dalpha, prob, dp, dbeta, st));
}

void run_alpha_from_prob(int dtype, int B, int H, int J, int K, const void* prob, const DropParams& dp, void* alpha,
                         hipStream_t st) {
    const int64_t n8 = (int64_t)B * H * J * K / 8;
    DM_DTYPE_SWITCH(dtype, hipLaunchKernelGGL((alpha_from_prob_k<T>), dim3((unsigned)((n8 + 255) / 256)), dim3(256), 0,
                                              st, n8, B, H, J, K, (const T*)prob, dp, (T*)alpha));
}

void run_ln_bwd(const LnBwdArgs& a, hipStream_t st) { DM_DTYPE_SWITCH(a.dtype, ln_bwd_t<T>(a, st)); }

void run_bias_act_fwd(int dtype, int64_t rows, int cols, const void* x, const void* bias, int act,
                      const DropParams& dp, void* y, hipStream_t st) {
    int64_t nvec = rows * cols / 8;
    DM_DTYPE_SWITCH(dtype, hipLaunchKernelGGL((bias_act_fwd_k<T>), dim3(grid_for(nvec)), dim3(NT), 0, st, nvec,
                                               cols, (const T*)x, (const T*)bias, act, dp, (T*)y));
}

void run_attn_input_bias(int dtype, int64_t rows, int H, int P, const void* x, const void* bq, const void* bk,
                         const void* bv, void* y, hipStream_t st) {
    int64_t nvec = rows * 3 * H * P / 8;
    DM_DTYPE_SWITCH(dtype, hipLaunchKernelGGL((attn_input_bias_k<T>), dim3(grid_for(nvec)), dim3(NT), 0, st,
                                               nvec, H, P, (const T*)x, (const T*)bq, (const T*)bk,
                                               (const T*)bv, (T*)y));
}

void run_act_bwd(int dtype, int64_t rows, int F, const void* da, const void* h, const void* b1, int act,
                 const DropParams& dp, void* dh, float* part, hipStream_t st, void* dht) {
    const int nblk = colsum_blocks(rows);
    if (dht) {
        // whole groups of 8 rows per block (the caller checked rows % 8 == 0)
        const int rpb = (int)((rows + nblk - 1) / nblk + 7) / 8 * 8;
        const int nrb = (int)((rows + rpb - 1) / rpb);
        const int ncb = (F / 8 + NT - 1) / NT;
        DM_DTYPE_SWITCH(dtype, hipLaunchKernelGGL((act_bwd_t_k<T>), dim3(nrb * ncb), dim3(NT), 0, st, rows, F,
                                                  (const T*)da, (const T*)h, (const T*)b1, act, dp, (T*)dh,
                                                  (T*)dht, part, rpb, nrb));
        // row blocks past nrb (up to colsum_blocks) would leave their
        // partial rows unwritten: the finish reads nrb rows (act_bwd_blocks)
        return;
    }
    const int rpb = (int)((rows + nblk - 1) / nblk);
    const dim3 grid(nblk, (F / 8 + NT - 1) / NT);
    DM_DTYPE_SWITCH(dtype, hipLaunchKernelGGL((act_bwd_k<T>), grid, dim3(NT), 0, st, rows, F, (const T*)da,
                                              (const T*)h, (const T*)b1, act, dp, (T*)dh, part, rpb));
}

void run_colsum_partial(int dtype, int64_t rows, int cols, const void* x, float* part, hipStream_t st) {
    const int nblk = colsum_blocks(rows);
    const int rpb = (int)((rows + nblk - 1) / nblk);
    const dim3 grid(nblk, (cols / 8 + NT - 1) / NT);
    DM_DTYPE_SWITCH(dtype, hipLaunchKernelGGL((colsum_partial_k<T>), grid, dim3(NT), 0, st, rows, cols,
                                              (const T*)x, part, rpb));
}

void run_colsum_finish_jobs(const FinishJob* jobs, int n, hipStream_t st) {
    FinishJobs fj{};
    fj.n = n;
    int blocks = 0;
    for (int i = 0; i < n; ++i) {
        fj.job[i] = jobs[i];
        fj.first[i] = blocks;
        blocks += (jobs[i].cols + FIN_COLS - 1) / FIN_COLS * jobs[i].nsets;
    }
    hipLaunchKernelGGL(colsum_finish_k, dim3(blocks), dim3(FIN_NT), 0, st, fj);
}

void run_colsum_finish(int nblk, int cols, const float* part, float* out, hipStream_t st) {
    const FinishJob j = finish_job(part, nblk, cols, out);
    run_colsum_finish_jobs(&j, 1, st);
}

void run_colsum_finish_qkv(int nblk, int H, int P, int nseg, const float* part, float* dbq, float* dbk,
                           float* dbv, hipStream_t st) {
    const FinishJob j = finish_job_qkv(part, nblk, H, P, nseg, dbq, dbk, dbv);
    run_colsum_finish_jobs(&j, 1, st);
}

void run_rowsum(int dtype, int64_t rows, int len, const void* x, float* out, hipStream_t st) {
    DM_DTYPE_SWITCH(dtype, hipLaunchKernelGGL((rowsum_k<T>), dim3((rows + 3) / 4), dim3(NT), 0, st, rows, len,
                                               (const T*)x, out));
}

void run_add(int dtype, int64_t n, const void* a, const void* b, void* out, hipStream_t st) {
    int64_t nvec = n / 8;
    DM_DTYPE_SWITCH(dtype, hipLaunchKernelGGL((add_k<T>), dim3(grid_for(nvec)), dim3(NT), 0, st, nvec,
                                               (const T*)a, (const T*)b, (T*)out));
}

void run_dropout_mask(const DropParams& dp, uint64_t offset, uint64_t n, uint8_t* out, hipStream_t st) {
    uint64_t nvec = n / 8;
    hipLaunchKernelGGL(dropout_mask_k, dim3(grid_for((int64_t)nvec)), dim3(NT), 0, st, dp, offset, nvec, out);
}

}  // namespace dm
