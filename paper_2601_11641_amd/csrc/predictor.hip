// Mask predictor kernels for gfx950 (wave64).
//
// All predictor arithmetic is fp64: the block sums of bf16 values are exact
// in fp64, and the statistic, the fit and the scores then agree with an fp64
// reference to rounding level, so the integer outcome (which blocks are kept)
// only depends on the float32 ranking keys.  Every reduction runs in a fixed
// order (no floating-point atomics), so results are bitwise reproducible.
//
// Paper references: block pooling + mass estimate stand in for the sparsity
// map of Eq. 2; the fit solves the normal equations of Eq. 4 with the block
// structure of Appendix B.4; the prediction is the linear extrapolation of
// Section 5.2; the selection implements the ranking and the gated
// block-diagonal support of Section 5.3.
#include "moddit_internal.h"

#include <cmath>

namespace moddit {
namespace {

constexpr int kThreads = 256;

__device__ inline double bf16_bits_to_double(uint32_t bits) {
    return static_cast<double>(__uint_as_float(bits << 16));
}

// Fixed-order tree reductions over one 256-thread workgroup.
__device__ double block_sum(double v, double* red) {
    red[threadIdx.x] = v;
    __syncthreads();
    for (int s = kThreads / 2; s > 0; s >>= 1) {
        if (threadIdx.x < s) red[threadIdx.x] += red[threadIdx.x + s];
        __syncthreads();
    }
    double r = red[0];
    __syncthreads();
    return r;
}

__device__ double block_max(double v, double* red) {
    red[threadIdx.x] = v;
    __syncthreads();
    for (int s = kThreads / 2; s > 0; s >>= 1) {
        if (threadIdx.x < s) red[threadIdx.x] = fmax(red[threadIdx.x], red[threadIdx.x + s]);
        __syncthreads();
    }
    double r = red[0];
    __syncthreads();
    return r;
}

// Exclusive scan over the 256 threads of a workgroup in thread order (a
// wave scan, then the wave totals added in wave order: a fixed order).
// wsum: kThreads / 64 entries of LDS scratch; *total receives the sum.
template <class T>
__device__ T block_exclusive_scan(T v, T* wsum, T* total) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    T incl = v;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const T y = __shfl_up(incl, off);
        if (lane >= off) incl += y;
    }
    if (lane == 63) wsum[w] = incl;
    __syncthreads();
    T base = T(0), all = T(0);
#pragma unroll
    for (int ww = 0; ww < kThreads / 64; ++ww) {
        if (ww < w) base += wsum[ww];
        all += wsum[ww];
    }
    __syncthreads();   // wsum may be reused by the caller
    *total = all;
    return base + (incl - v);
}

// In-place inclusive prefix sum of a[0 .. len) in LDS over one work-group:
// thread t scans its contiguous segment, the segment totals are scanned in
// thread order, and each segment adds its offset (a fixed order).  Every
// thread of the work-group calls it; a is complete on return.
__device__ void block_inclusive_prefix(double* a, int len, double* wsum) {
    const int seg = (len + kThreads - 1) / kThreads;
    const int b0 = min(len, (int)threadIdx.x * seg), b1 = min(len, b0 + seg);
    double run = 0.0;
    for (int b = b0; b < b1; ++b) {
        run += a[b];
        a[b] = run;
    }
    double total;
    const double off = block_exclusive_scan<double>(run, wsum, &total);
    for (int b = b0; b < b1; ++b) a[b] += off;
    __syncthreads();
}

// ---------------------------------------------------------------------------
// a1: block pooling.  Grid (n, BH, 2): z = 0 pools Q, z = 1 pools K.  The
// block is one contiguous run of rows*D bf16.  Lane l of wave w reads the
// 16-byte chunk l % C (C = D / 8 chunks per row) of rows p*RPP + w*RPW +
// l / C of every pass p; all of a thread's loads (non-temporal) are issued
// before any is used (the whole 32 KB block in flight per work-group), and
// accumulated in fp64.  The rows of a wave are then folded with lane shuffles (xor C, 2C,
// ...), the four waves' sums through LDS in wave order: a fixed summation
// order.  L: tokens pooled (the video tokens); L_stride: tokens per head in
// memory.
// ---------------------------------------------------------------------------
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

template <int D, int BS>
__global__ __launch_bounds__(kThreads) void pool_kernel(const uint16_t* __restrict__ q,
                                                        const uint16_t* __restrict__ k,
                                                        double* __restrict__ qbar,
                                                        double* __restrict__ kbar, int L,
                                                        int L_stride, int n) {
    constexpr int C = D / 8;               // 16-byte chunks per row
    constexpr int NW = kThreads / 64;      // waves
    constexpr int RPW = 64 / C;            // rows per wave per pass
    constexpr int RPP = NW * RPW;          // rows per pass
    constexpr int NP = BS / RPP;           // passes
    static_assert(BS % RPP == 0, "block rows must fill whole passes");
    __shared__ double part[NW][D];
    const int i = blockIdx.x, bh = blockIdx.y;
    const uint16_t* src = (blockIdx.z == 0 ? q : k) + ((size_t)bh * L_stride + (size_t)i * BS) * D;
    double* dst = (blockIdx.z == 0 ? qbar : kbar) + ((size_t)bh * n + i) * D;
    const int cnt = min(BS, L - i * BS);
    const int t = threadIdx.x, lane = t & 63, w = t >> 6, c = lane % C, rs = lane / C;
    uint4 v[NP];
#pragma unroll
    for (int p = 0; p < NP; ++p) {
        const int r = p * RPP + w * RPW + rs;
        // read once and never again: non-temporal loads keep the stream out of the caches
        v[p] = r < cnt ? __builtin_bit_cast(uint4, __builtin_nontemporal_load(
                             reinterpret_cast<const u32x4*>(src + (size_t)r * D + c * 8)))
                       : make_uint4(0, 0, 0, 0);
    }
    double acc[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] = 0.0;
#pragma unroll
    for (int p = 0; p < NP; ++p) {
        const uint32_t ws[4] = {v[p].x, v[p].y, v[p].z, v[p].w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            acc[2 * e] += bf16_bits_to_double(ws[e] & 0xFFFFu);
            acc[2 * e + 1] += bf16_bits_to_double(ws[e] >> 16);
        }
    }
#pragma unroll
    for (int off = C; off < 64; off <<= 1)
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[e] += __shfl_xor(acc[e], off);
    if (rs == 0) {
#pragma unroll
        for (int e = 0; e < 8; ++e) part[w][c * 8 + e] = acc[e];
    }
    __syncthreads();
    if (t < D) {
        double sum = 0.0;
#pragma unroll
        for (int ww = 0; ww < NW; ++ww) sum += part[ww][t];
        dst[t] = sum / static_cast<double>(cnt);
    }
}

// ---------------------------------------------------------------------------
// a2 (part 1): block logits scale * qbar_i . kbar_j with fp64 matrix
// products (v_mfma_f64_16x16x4_f64): a 128 x 128 tile per work-group, 64 x 64
// per wave (4 x 4 product tiles of 16 x 16), channels staged through LDS 16
// at a time.  Operand layout of the product (16 x 4 times 4 x 16): lane l
// supplies A[l % 16][l / 16] and B[l / 16][l % 16], and holds D[l / 16 + 4 e]
// [l % 16] in element e of its result.
// ---------------------------------------------------------------------------
typedef double f64x4 __attribute__((ext_vector_type(4)));

template <int D>
__global__ __launch_bounds__(kThreads) void logits_kernel(const double* __restrict__ qbar,
                                                          const double* __restrict__ kbar,
                                                          double* __restrict__ G, int n,
                                                          double scale) {
    constexpr int T = 128, KC = 16;
    static_assert(D % KC == 0 && kThreads == 256, "four waves, 16-channel chunks");
    __shared__ double qs[T][KC + 1];
    __shared__ double ks[T][KC + 1];
    const int bh = blockIdx.z, i0 = blockIdx.y * T, j0 = blockIdx.x * T;
    const double* qb = qbar + (size_t)bh * n * D;
    const double* kb = kbar + (size_t)bh * n * D;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int wr = (w >> 1) * 64, wc = (w & 1) * 64;   // the wave's 64 x 64 sub-tile
    const int lm = lane & 15, lk = lane >> 4;
    f64x4 acc[4][4];
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int v = 0; v < 4; ++v) acc[u][v] = f64x4{0.0, 0.0, 0.0, 0.0};
    // the next chunk is loaded into registers while this one is multiplied
    constexpr int PT = T * KC / kThreads;   // values of each operand per thread
    double qn[PT], kn[PT];
    auto fetch = [&](int d0) {
#pragma unroll
        for (int x = 0; x < PT; ++x) {
            const int e = threadIdx.x + x * kThreads, r = e / KC, c = e % KC;
            qn[x] = (i0 + r < n) ? qb[(size_t)(i0 + r) * D + d0 + c] : 0.0;
            kn[x] = (j0 + r < n) ? kb[(size_t)(j0 + r) * D + d0 + c] : 0.0;
        }
    };
    fetch(0);
    for (int d0 = 0; d0 < D; d0 += KC) {
#pragma unroll
        for (int x = 0; x < PT; ++x) {
            const int e = threadIdx.x + x * kThreads, r = e / KC, c = e % KC;
            qs[r][c] = qn[x];
            ks[r][c] = kn[x];
        }
        __syncthreads();
        if (d0 + KC < D) fetch(d0 + KC);
#pragma unroll
        for (int kk = 0; kk < KC; kk += 4) {
            double a[4], b[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                a[u] = qs[wr + 16 * u + lm][kk + lk];
                b[u] = ks[wc + 16 * u + lm][kk + lk];
            }
#pragma unroll
            for (int u = 0; u < 4; ++u)
#pragma unroll
                for (int v = 0; v < 4; ++v)
                    acc[u][v] = __builtin_amdgcn_mfma_f64_16x16x4f64(a[u], b[v], acc[u][v], 0, 0, 0);
        }
        __syncthreads();
    }
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int i = i0 + wr + 16 * u + lk + 4 * e;
            if (i >= n) continue;
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int j = j0 + wc + 16 * v + lm;
                if (j < n) G[((size_t)bh * n + i) * n + j] = scale * acc[u][v][e];
            }
        }
}

// ---------------------------------------------------------------------------
// a2 (part 2): G(i, j) = |j| exp(l_ij - max_j l) / sum_j |j| exp(...), one
// workgroup per (head, row), in place.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kThreads) void mass_softmax_kernel(double* __restrict__ G, int L,
                                                                int bs, int n) {
    constexpr int NPT = kMaxBlocks / kThreads;   // row entries per thread at most
    __shared__ double red[kThreads];
    double* g = G + (size_t)blockIdx.x * n;
    // the row is read once into registers (entry j = threadIdx.x + c kThreads)
    double x[NPT];
    double m = -INFINITY;
#pragma unroll
    for (int c = 0; c < NPT; ++c) {
        const int j = threadIdx.x + c * kThreads;
        x[c] = j < n ? g[j] : -INFINITY;
        m = fmax(m, x[c]);
    }
    m = block_max(m, red);
    double s = 0.0;
#pragma unroll
    for (int c = 0; c < NPT; ++c) {
        const int j = threadIdx.x + c * kThreads;
        if (j < n) {
            x[c] = static_cast<double>(min(bs, L - j * bs)) * exp(x[c] - m);
            s += x[c];
        }
    }
    s = block_sum(s, red);
#pragma unroll
    for (int c = 0; c < NPT; ++c) {
        const int j = threadIdx.x + c * kThreads;
        if (j < n) g[j] = x[c] / s;
    }
}

// ---------------------------------------------------------------------------
// a3 (rhs): r = M^T vec(G): diagonal sums (2n-1), column sums (n) and frame
// square sums (F).  Diagonals and columns: the rows split into kRhsChunks
// fixed ranges; per (output, range) one thread takes the range's entries in
// row order into four interleaved partial sums (rows i mod 4) combined as
// (s0 + s1) + (s2 + s3), consecutive threads reading consecutive addresses;
// the ranges' sums are then added in range order.  Frame squares: one
// work-group per (frame, head), a fixed assignment of entries to threads and
// a fixed-order tree.  Every sum has a fixed order, so the result is
// deterministic.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kThreads) void rhs_kernel(const double* __restrict__ G,
                                                       double* __restrict__ part, int BH, int n) {
    const int bh = blockIdx.z, ch = blockIdx.y;
    const int o = blockIdx.x * kThreads + threadIdx.x;
    if (o >= 3 * n - 1) return;
    const double* g = G + (size_t)bh * n * n;
    // rows [ch n / kRhsChunks, (ch + 1) n / kRhsChunks) of the output's entries
    const int r0 = (int)((long long)ch * n / kRhsChunks), r1 = (int)((long long)(ch + 1) * n / kRhsChunks) - 1;
    int i0, i1;
    size_t step, at;
    if (o < 2 * n - 1) {                 // diagonal j - i = dl
        const int dl = o - (n - 1);
        i0 = max(r0, max(0, -dl));
        i1 = min(r1, min(n - 1, n - 1 - dl));
        step = (size_t)n + 1;
        at = (size_t)i0 * n + i0 + dl;
    } else {                             // column j
        i0 = r0;
        i1 = r1;
        step = (size_t)n;
        at = (size_t)i0 * n + (o - (2 * n - 1));
    }
    double s0 = 0.0, s1 = 0.0, s2 = 0.0, s3 = 0.0;
    int i = i0;
    for (; i + 3 <= i1; i += 4, at += 4 * step) {
        s0 += g[at];
        s1 += g[at + step];
        s2 += g[at + 2 * step];
        s3 += g[at + 3 * step];
    }
    for (int q = 0; i <= i1; ++i, ++q, at += step) {
        if (q == 0) s0 += g[at];
        else if (q == 1) s1 += g[at];
        else s2 += g[at];
    }
    part[((size_t)ch * BH + bh) * (3 * n - 1) + o] = (s0 + s1) + (s2 + s3);
}

// The ranges' sums of every diagonal and column, added in range order.
__global__ __launch_bounds__(kThreads) void rhs_sum_kernel(const double* __restrict__ part,
                                                           double* __restrict__ r, int BH, int n, int F) {
    const int bh = blockIdx.y;
    const int o = blockIdx.x * kThreads + threadIdx.x;
    if (o >= 3 * n - 1) return;
    double s = part[(size_t)bh * (3 * n - 1) + o];
#pragma unroll
    for (int ch = 1; ch < kRhsChunks; ++ch) s += part[((size_t)ch * BH + bh) * (3 * n - 1) + o];
    r[(size_t)bh * (3 * n - 1 + F) + o] = s;
}

__global__ __launch_bounds__(kThreads) void rhs_frame_kernel(const double* __restrict__ G,
                                                             const int* __restrict__ reg,
                                                             double* __restrict__ r, int n, int F) {
    __shared__ double red[kThreads];
    const int f = blockIdx.x, bh = blockIdx.y;
    const int lo = reg[2 * f], hi = reg[2 * f + 1], sz = hi - lo + 1;
    const double* g = G + (size_t)bh * n * n;
    double s = 0.0;
    for (int e = threadIdx.x; e < sz * sz; e += kThreads) s += g[(size_t)(lo + e / sz) * n + lo + e % sz];
    s = block_sum(s, red);
    if (threadIdx.x == 0) r[(size_t)bh * (3 * n - 1 + F) + 3 * n - 1 + f] = s;
}

// ---------------------------------------------------------------------------
// a3 (solve).  The normal matrix N = M^T M has a diagonal C^T C block
// (Appendix B.4).  Fixing the gauge by dropping the last vertical column,
// the unknowns split into c (2n-1) and u = [d_0..d_{n-2}, e] (q = n-1+F):
//   [Dc  W ] [c]   [r_C]          S = Y - W^T Dc^{-1} W   (host, inverted)
//   [W^T Y ] [u] = [r_U],         u = S^{-1} (r_U - W^T Dc^{-1} r_C)
//                                 c = Dc^{-1} (r_C - W u)
// with Dc = diag(n - |delta|), W[delta, j] = 1 iff column j crosses
// diagonal delta, W[delta, f] = max(0, |R_f| - |delta|).  The result is
// moved to the minimum-norm gauge by removing its component along
// z = [1, -1, 0].
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kThreads) void solve_pre_kernel(const double* __restrict__ r,
                                                             const int* __restrict__ reg,
                                                             double* __restrict__ bU, int n,
                                                             int F) {
    extern __shared__ double y[];   // 2n - 1: Dc^{-1} r_C, then its inclusive prefix
    __shared__ double wsum[kThreads / 64];
    const int bh = blockIdx.y;      // x: a chunk of kThreads outputs
    const int p = 3 * n - 1 + F, q = n - 1 + F;
    const double* rr = r + (size_t)bh * p;
    for (int a = threadIdx.x; a < 2 * n - 1; a += kThreads)
        y[a] = rr[a] / static_cast<double>(n - abs(a - (n - 1)));
    __syncthreads();
    const int j = blockIdx.x * kThreads + threadIdx.x;
    // frame rows of W^T: weighted sums of the diagonals a frame square spans
    double s = 0.0;
    if (j >= n - 1 && j < q) {
        const int f = j - (n - 1);
        const int sz = reg[2 * f + 1] - reg[2 * f] + 1;
        for (int dl = -(sz - 1); dl <= sz - 1; ++dl)
            s += static_cast<double>(sz - abs(dl)) * y[dl + n - 1];
    }
    __syncthreads();
    // column rows of W^T: the n diagonals column j crosses, y[j .. j + n - 1],
    // as a difference of the prefix sums
    block_inclusive_prefix(y, 2 * n - 1, wsum);
    if (j < n - 1) s = y[j + n - 1] - (j > 0 ? y[j - 1] : 0.0);
    if (j < q) bU[(size_t)bh * q + j] = (j < n - 1 ? rr[2 * n - 1 + j] : rr[3 * n - 1 + (j - (n - 1))]) - s;
}

// u[h] = S^{-1} bU[h] for all heads, split over kSolveSplit fixed chunks of
// k: part[c][h][j] = sum over k in chunk c (ascending) of S^{-1}[k][j] bU[h][k]
// (S^{-1} symmetric, read row-wise: a wave's lanes read 64 consecutive
// columns).  The post kernel adds the chunks in order, so the result does
// not depend on the launch.  Grid: (column chunks of 64, kSolveSplit); wave
// w takes heads w*8.. in passes of 32.
__global__ __launch_bounds__(kThreads) void solve_gemv_kernel(const double* __restrict__ Sinv,
                                                              const double* __restrict__ bU,
                                                              double* __restrict__ part, int q,
                                                              int BH) {
    constexpr int HW = 8;
    // a wave's right-hand sides, 64 k at a time: bs[w][k - kb][hh]
    __shared__ double bs[kThreads / 64][64][HW];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int j = blockIdx.x * 64 + lane;
    const int c = blockIdx.y;
    const int kc = (q + kSolveSplit - 1) / kSolveSplit;
    const int k0 = min(q, c * kc), k1 = min(q, k0 + kc);
    for (int h0 = w * HW; h0 < BH; h0 += (kThreads / 64) * HW) {
        double acc[HW];
#pragma unroll
        for (int hh = 0; hh < HW; ++hh) acc[hh] = 0.0;
        for (int kb = k0; kb < k1; kb += 64) {
            const int kn = min(64, k1 - kb);
            // (the wave's LDS operations run in order: the previous pass's
            // reads are done before these writes)
#pragma unroll
            for (int hh = 0; hh < HW; ++hh)
                bs[w][lane][hh] = (lane < kn && h0 + hh < BH) ? bU[(size_t)(h0 + hh) * q + kb + lane] : 0.0;
            if (j < q) {
#pragma unroll 4
                for (int kk = 0; kk < kn; ++kk) {
                    const double a = Sinv[(size_t)(kb + kk) * q + j];
#pragma unroll
                    for (int hh = 0; hh < HW; ++hh) acc[hh] = fma(a, bs[w][kk][hh], acc[hh]);
                }
            }
        }
        if (j < q) {
#pragma unroll
            for (int hh = 0; hh < HW; ++hh)
                if (h0 + hh < BH) part[((size_t)c * BH + h0 + hh) * q + j] = acc[hh];
        }
    }
}

__global__ __launch_bounds__(kThreads) void solve_post_kernel(const double* __restrict__ r,
                                                              const double* __restrict__ u,
                                                              const int* __restrict__ reg,
                                                              double* __restrict__ X, int n,
                                                              int F, int BH) {
    extern __shared__ double us[];   // q: u, then the prefix of its first n - 1 entries; then F frame sizes
    __shared__ double wsum[kThreads / 64];
    __shared__ int szmax;
    const int bh = blockIdx.x;       // one work-group per head
    const int p = 3 * n - 1 + F, q = n - 1 + F;
    int* sz = reinterpret_cast<int*>(us + q);
    if (threadIdx.x == 0) szmax = 0;
    __syncthreads();
    for (int f = threadIdx.x; f < F; f += kThreads) {
        sz[f] = reg[2 * f + 1] - reg[2 * f] + 1;
        atomicMax(&szmax, sz[f]);
    }
    const double* rr = r + (size_t)bh * p;
    double* x = X + (size_t)bh * p;
    // u = sum of the k-chunk partial products, in chunk order; the d and e
    // parts of X are u itself
    for (int a = threadIdx.x; a < q; a += kThreads) {
        double v = 0.0;
        for (int c = 0; c < kSolveSplit; ++c) v += u[((size_t)c * BH + bh) * q + a];
        us[a] = v;
        if (a < n - 1) x[2 * n - 1 + a] = v;
        else x[3 * n - 1 + (a - (n - 1))] = v;
    }
    if (threadIdx.x == 0) x[3 * n - 2] = 0.0;   // d_{n-1}: the gauge column dropped
    __syncthreads();
    block_inclusive_prefix(us, n - 1, wsum);
    // c = Dc^{-1} (r_C - W u): the columns crossing diagonal dl are a window
    // of d (a difference of the prefix sums), the frames' weights max(0,
    // |R_f| - |dl|) multiply e
    for (int a = threadIdx.x; a < 2 * n - 1; a += kThreads) {
        const int dl = a - (n - 1);
        const int j0 = max(0, dl), j1 = min(n - 2, dl + n - 1);
        double s = j1 >= j0 ? us[j1] - (j0 > 0 ? us[j0 - 1] : 0.0) : 0.0;
        if (abs(dl) < szmax) {   // only diagonals shorter than a frame square's side meet one
            for (int f = 0; f < F; ++f) {
                const int w = sz[f] - abs(dl);
                if (w > 0) s += static_cast<double>(w) * us[n - 1 + f];
            }
        }
        x[a] = (rr[a] - s) / static_cast<double>(n - abs(dl));
    }
}

// Minimum-norm gauge: remove the component of X along z = [1, -1, 0].
__global__ __launch_bounds__(kThreads) void solve_gauge_kernel(double* __restrict__ X, int n, int F) {
    __shared__ double red[kThreads];
    const int p = 3 * n - 1 + F;
    double* x = X + (size_t)blockIdx.x * p;
    double part = 0.0;   // sum(c) - sum(d) of this thread's entries
    for (int a = threadIdx.x; a < 2 * n - 1; a += kThreads) part += x[a];
    for (int j = threadIdx.x; j < n; j += kThreads) part -= x[2 * n - 1 + j];
    const double alpha = block_sum(part, red) / static_cast<double>(3 * n - 1);
    for (int a = threadIdx.x; a < 2 * n - 1; a += kThreads) x[a] -= alpha;
    for (int j = threadIdx.x; j < n; j += kThreads) x[2 * n - 1 + j] += alpha;
}

// ---------------------------------------------------------------------------
// Gate: on iff min over the anchors of the frame-averaged e exceeds tau_e.
// ---------------------------------------------------------------------------
__global__ void gate_kernel(const double* __restrict__ Xa, const double* __restrict__ Xb,
                            int32_t* __restrict__ gate, int BH, int n, int F, double tau_e) {
    const int bh = blockIdx.x * blockDim.x + threadIdx.x;
    if (bh >= BH) return;
    const int p = 3 * n - 1 + F;
    double ea = 0.0, eb = 0.0;
    for (int f = 0; f < F; ++f) {
        ea += Xa[(size_t)bh * p + 3 * n - 1 + f];
        eb += Xb[(size_t)bh * p + 3 * n - 1 + f];
    }
    ea /= F;
    eb /= F;
    gate[bh] = fmin(ea, eb) > tau_e ? 1 : 0;
}

// ---------------------------------------------------------------------------
// a4: linear extrapolation of c and d (Section 5.2).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kThreads) void extrapolate_kernel(const double* __restrict__ X1,
                                                               const double* __restrict__ X2,
                                                               double w,
                                                               double* __restrict__ pred,
                                                               int n, int F) {
    const int bh = blockIdx.y;
    const int a = blockIdx.x * kThreads + threadIdx.x;
    const int m = 3 * n - 1, p = 3 * n - 1 + F;
    if (a >= m) return;
    const double x2 = X2[(size_t)bh * p + a], x1 = X1[(size_t)bh * p + a];
    pred[(size_t)bh * m + a] = x2 + (x2 - x1) * w;
}

// ---------------------------------------------------------------------------
// a5: per-row selection.  One wave per (head, query block i) up to n = 1024
// (select_wave_kernel), one work-group of 256 threads per row above
// (select_kernel), both by the same threshold search.
//   sigma_j = n (c~[j-i] + d~[j]) in fp64, rounded to float: the ranking key.
//   The non-forced blocks are ranked by (sigma desc, j asc).  TOPK keeps the
//   first max(0, k - |forced|) of them; MASS keeps the shortest prefix whose
//   positive key mass, added to the forced blocks' mass, reaches tau of the
//   row total (fp64 sums; at least one block).  The kept set is compacted in
//   ascending j.
// With a text segment after the video (token-type-aware masking) n counts
// the video blocks, the lists have ldn >= n entries per row, the block tb0
// shared by the video and the text (tb0 < n) is forced, and every row keeps
// the text blocks n .. ldn-1 after its video selection.  tb0 >= ldn: none.
// ---------------------------------------------------------------------------
__device__ inline uint32_t order_bits(float f) {
    const uint32_t u = __float_as_uint(f);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ inline float order_bits_to_float(uint32_t k) {
    const uint32_t u = (k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k;
    return __uint_as_float(u);
}

// The wave's total of a per-lane double in a fixed order, the same bits in
// every lane: sums within rows of 16 lanes by DPP (lane pairs, quad pairs,
// then rotations by 4 and 8, after which lane 0 of a row holds its row's
// sum), then the four row sums read from lanes 0, 16, 32 and 48.
__device__ inline double dpp_f64(double v, int ctrl_id) {
    const uint64_t u = __builtin_bit_cast(uint64_t, v);
    uint32_t lo = static_cast<uint32_t>(u), hi = static_cast<uint32_t>(u >> 32);
    switch (ctrl_id) {
        case 0: lo = __builtin_amdgcn_mov_dpp((int)lo, 0xB1, 0xF, 0xF, false);
                hi = __builtin_amdgcn_mov_dpp((int)hi, 0xB1, 0xF, 0xF, false); break;   // quad_perm 1,0,3,2
        case 1: lo = __builtin_amdgcn_mov_dpp((int)lo, 0x4E, 0xF, 0xF, false);
                hi = __builtin_amdgcn_mov_dpp((int)hi, 0x4E, 0xF, 0xF, false); break;   // quad_perm 2,3,0,1
        case 2: lo = __builtin_amdgcn_mov_dpp((int)lo, 0x124, 0xF, 0xF, false);
                hi = __builtin_amdgcn_mov_dpp((int)hi, 0x124, 0xF, 0xF, false); break;  // row_ror:4
        default: lo = __builtin_amdgcn_mov_dpp((int)lo, 0x128, 0xF, 0xF, false);
                 hi = __builtin_amdgcn_mov_dpp((int)hi, 0x128, 0xF, 0xF, false); break; // row_ror:8
    }
    return __builtin_bit_cast(double, (static_cast<uint64_t>(hi) << 32) | lo);
}

__device__ inline double readlane_f64(double v, int l) {
    const uint64_t u = __builtin_bit_cast(uint64_t, v);
    const uint32_t lo = __builtin_amdgcn_readlane(static_cast<uint32_t>(u), l);
    const uint32_t hi = __builtin_amdgcn_readlane(static_cast<uint32_t>(u >> 32), l);
    return __builtin_bit_cast(double, (static_cast<uint64_t>(hi) << 32) | lo);
}

__device__ inline double wave_total_f64(double v) {
    v += dpp_f64(v, 0);
    v += dpp_f64(v, 1);
    v += dpp_f64(v, 2);
    v += dpp_f64(v, 3);
    return (readlane_f64(v, 0) + readlane_f64(v, 16)) + (readlane_f64(v, 32) + readlane_f64(v, 48));
}

// The same selection with one 256-thread work-group per row (n <= 256 E),
// E keys per thread (blocks t + 256 e, coalesced), by the threshold search of
// select_wave_kernel below: each step's count or fp64 sum is taken per wave
// (scalar counts of 64-lane masks; the fixed-order wave total) and over the
// four waves in wave order, so every thread holds the same bits.
template <int E>
__global__ __launch_bounds__(kThreads) void select_kernel(
    const double* __restrict__ pred, const int32_t* __restrict__ gate,
    const int* __restrict__ row_lo, const int* __restrict__ row_hi, int mode, int topk,
    double tau, int32_t* __restrict__ kv_idx, int32_t* __restrict__ kv_cnt, int n,
    int ldn, int tb0) {
    constexpr int NW = kThreads / 64;
    static_assert(NW == 4, "the wave totals are added as (w0 + w1) + (w2 + w3)");
    extern __shared__ __align__(16) unsigned char smem[];
    int* flag = reinterpret_cast<int*>(smem);                     // npad
    __shared__ double wsum_d[NW];
    __shared__ int wsum_i[NW];

    const int row = blockIdx.x;
    const int bh = row / n, i = row % n;
    const double* c = pred + (size_t)bh * (3 * n - 1);
    const double* d = c + (2 * n - 1);
    const bool g = gate[bh] != 0;
    const int flo = row_lo[i], fhi = row_hi[i];
    // forced: the frame blocks of i (gate on) and the block shared by the
    // video and the text segment (tb0 < n), which is a text block
    const bool tb_in_frames = g && tb0 >= flo && tb0 <= fhi;
    const int nf = (g ? (fhi - flo + 1) : 0) + ((tb0 < n && !tb_in_frames) ? 1 : 0);
    const int n_free = n - nf;
    const int t = threadIdx.x, lane = t & 63, w = t >> 6;

    double forced_mass = 0.0;
    uint32_t vb[E];
    double ms[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
        const int j = t + kThreads * e;   // coalesced
        vb[e] = 0;
        ms[e] = 0.0;
        int fl = 0;
        if (j < n) {
            const double sv = static_cast<double>(n) * (c[j - i + n - 1] + d[j]);
            const float kf = static_cast<float>(sv);
            if ((g && j >= flo && j <= fhi) || j == tb0) {
                fl = 1;
                forced_mass += fmax(static_cast<double>(kf), 0.0);
            } else {
                vb[e] = order_bits(kf);
                ms[e] = fmax(static_cast<double>(kf), 0.0);
            }
        }
        flag[j] = fl;
    }
    auto total_f64 = [&](double v) {    // over the work-group, fixed order
        v = wave_total_f64(v);
        if (lane == 0) wsum_d[w] = v;
        __syncthreads();
        const double tot = (wsum_d[0] + wsum_d[1]) + (wsum_d[2] + wsum_d[3]);
        __syncthreads();
        return tot;
    };
    auto count_ge = [&](uint32_t th) {  // free keys with bits >= th (th >= 1)
        int cnt = 0;
#pragma unroll
        for (int e = 0; e < E; ++e) cnt += __popcll(__ballot(vb[e] >= th));
        if (lane == 0) wsum_i[w] = cnt;
        __syncthreads();
        const int tot = (wsum_i[0] + wsum_i[1]) + (wsum_i[2] + wsum_i[3]);
        __syncthreads();
        return tot;
    };
    auto mass_ge = [&](uint32_t th) {   // their mass (th >= 1)
        double sm = 0.0;
#pragma unroll
        for (int e = 0; e < E; ++e) sm += vb[e] >= th ? ms[e] : 0.0;
        return total_f64(sm);
    };

    uint32_t p;     // boundary bits
    int r;          // keys kept at the boundary, in ascending j
    int keep = -1;  // free keys kept, when found by count
    if (mode == 0) {
        keep = min(n_free, max(0, topk - nf));
    } else {
        const double fm = total_f64(forced_mass);
        const double total = fm + (n_free > 0 ? mass_ge(1u) : 0.0);
        const double target = tau * total;
        const int kmin = nf > 0 ? 0 : 1;
        if (fm >= target) {
            keep = min(n_free, kmin);
        } else if (total < target) {
            keep = n_free;
        } else {
            p = 0x80000000u;   // the boundary key has a positive mass
            for (int b = 30; b >= 0; --b) {
                const uint32_t th = p | (1u << b);
                if (fm + mass_ge(th) >= target) p = th;
            }
            const double hi = fm + (p < 0xFFFFFFFFu ? mass_ge(p + 1) : 0.0);
            const int ties = count_ge(p) - (p < 0xFFFFFFFFu ? count_ge(p + 1) : 0);
            const double mp = fmax(static_cast<double>(order_bits_to_float(p)), 0.0);
            r = 1;
            while (r < ties && hi + static_cast<double>(r) * mp < target) ++r;
        }
    }
    if (keep >= 0) {
        if (keep == 0) {
            p = 0xFFFFFFFFu;
            r = 0;
        } else if (keep >= n_free) {
            p = 0;
            r = 0;
        } else {
            p = 0;
            for (int b = 31; b >= 0; --b) {
                const uint32_t th = p | (1u << b);
                if (count_ge(th) >= keep) p = th;
            }
            r = keep - (p < 0xFFFFFFFFu ? count_ge(p + 1) : 0);
        }
    }
    // flags: 1 kept, 2 at the boundary (resolved below in ascending j)
#pragma unroll
    for (int e = 0; e < E; ++e) {
        const int j = t + kThreads * e;
        if (vb[e] > p)
            flag[j] = 1;
        else if (vb[e] == p && vb[e] != 0)
            flag[j] = 2;
    }
    __syncthreads();
    int f[E];
    int nt = 0;
#pragma unroll
    for (int e = 0; e < E; ++e) {
        f[e] = flag[t * E + e];
        nt += f[e] == 2;
    }
    int ntie;
    int tr = block_exclusive_scan(nt, wsum_i, &ntie);   // boundary keys before this thread
    int cnt = 0;
#pragma unroll
    for (int e = 0; e < E; ++e) {
        if (f[e] == 2) f[e] = tr++ < r ? 1 : 0;
        cnt += f[e];
    }

    // compaction in ascending j
    int total;
    int pos = block_exclusive_scan(cnt, wsum_i, &total);
    const size_t orow = (size_t)bh * ldn + i;     // row of the [BH, ldn, ldn] lists
    int32_t* out = kv_idx + orow * ldn;
#pragma unroll
    for (int e = 0; e < E; ++e) {
        const int j = t * E + e;
        if (f[e]) out[pos++] = j;
    }
    // text blocks after the video blocks: kept in every row
    for (int j = n + t; j < ldn; j += kThreads) out[total + (j - n)] = j;
    if (t == 0) kv_cnt[orow] = total + (ldn - n);
}

template <class T>
__device__ inline T wave_inclusive_scan(T v, int lane) {
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const T y = __shfl_up(v, off);
        if (lane >= off) v += y;
    }
    return v;
}

__device__ inline void wave_sync_lds() {
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    __builtin_amdgcn_wave_barrier();
}

// One wave per row (n <= 64 EW).  Every free block j holds its ranking key
// as the order bits of sigma_j (vb, 0 for forced blocks and padding) and its
// positive mass.  The kept free blocks are those whose bits exceed a
// boundary p, plus the first r in ascending j of those whose bits equal p:
// the same set as the first keep entries of the (sigma desc, j asc) order.
//   TOPK: p is the largest 32-bit value with at least keep free keys at or
//     above it (built bit by bit from the top, 32 wave-wide counts).
//   MASS: p is the largest value whose keys at or above it, added to the
//     forced mass, reach tau of the row total (31 fixed-order fp64 wave
//     sums below the sign bit, which a key of positive mass has set); every
//     key above p is needed, and r is the fewest keys at p
//     (all of mass max(sigma_p, 0)) that reach the target with them.
template <int EW>
__global__ __launch_bounds__(kThreads) void select_wave_kernel(
    const double* __restrict__ pred, const int32_t* __restrict__ gate,
    const int* __restrict__ row_lo, const int* __restrict__ row_hi, int mode, int topk,
    double tau, int32_t* __restrict__ kv_idx, int32_t* __restrict__ kv_cnt, int n,
    int ldn, int tb0, int rows) {
    constexpr int npad = 64 * EW;
    constexpr int WPG = kThreads / 64;
    __shared__ uint8_t flags[WPG][npad];
    const int lane = threadIdx.x & 63;
    const int wv = threadIdx.x >> 6;
    const int row = blockIdx.x * WPG + wv;        // wave-uniform
    if (row >= rows) return;
    uint8_t* flag = flags[wv];

    const int bh = row / n, i = row % n;
    const double* c = pred + (size_t)bh * (3 * n - 1);
    const double* d = c + (2 * n - 1);
    const bool g = gate[bh] != 0;
    const int flo = row_lo[i], fhi = row_hi[i];
    const bool tb_in_frames = g && tb0 >= flo && tb0 <= fhi;
    const int nf = (g ? (fhi - flo + 1) : 0) + ((tb0 < n && !tb_in_frames) ? 1 : 0);
    const int n_free = n - nf;

    double forced_mass = 0.0;
    uint32_t vb[EW];
    double ms[EW];
#pragma unroll
    for (int e = 0; e < EW; ++e) {
        const int j = lane + 64 * e;   // coalesced
        vb[e] = 0;
        ms[e] = 0.0;
        uint8_t fl = 0;
        if (j < n) {
            const double sv = static_cast<double>(n) * (c[j - i + n - 1] + d[j]);
            const float kf = static_cast<float>(sv);
            if ((g && j >= flo && j <= fhi) || j == tb0) {
                fl = 1;
                forced_mass += fmax(static_cast<double>(kf), 0.0);
            } else {
                vb[e] = order_bits(kf);
                ms[e] = fmax(static_cast<double>(kf), 0.0);
            }
        }
        flag[j] = fl;
    }
    auto count_ge = [&](uint32_t th) {   // free keys with bits >= th (th >= 1)
        int cnt = 0;
#pragma unroll
        for (int e = 0; e < EW; ++e) cnt += __popcll(__ballot(vb[e] >= th));
        return cnt;
    };
    auto mass_ge = [&](uint32_t th) {    // their mass (th >= 1)
        double s = 0.0;
#pragma unroll
        for (int e = 0; e < EW; ++e) s += vb[e] >= th ? ms[e] : 0.0;
        return wave_total_f64(s);
    };
    // largest p with count_ge(p) >= kk (kk >= 1, at most n_free)
    auto kth_bits = [&](int kk) {
        uint32_t p = 0;
        for (int b = 31; b >= 0; --b) {
            const uint32_t th = p | (1u << b);
            if (count_ge(th) >= kk) p = th;
        }
        return p;
    };

    uint32_t p;   // boundary bits
    int r;        // keys kept at the boundary, in ascending j
    int keep = -1;  // free keys kept when all or none are
    if (mode == 0) {
        keep = min(n_free, max(0, topk - nf));
    } else {
        const double fm = wave_total_f64(forced_mass);
        const double total = fm + (n_free > 0 ? mass_ge(1u) : 0.0);
        const double target = tau * total;
        const int kmin = nf > 0 ? 0 : 1;
        if (fm >= target) {
            keep = min(n_free, kmin);
        } else if (total < target) {
            keep = n_free;
        } else {
            // the boundary key has a positive mass, so its sign bit is set
            // (every non-negative key's mass is the total's free part)
            p = 0x80000000u;
            for (int b = 30; b >= 0; --b) {
                const uint32_t th = p | (1u << b);
                if (fm + mass_ge(th) >= target) p = th;
            }
            const double hi = fm + (p < 0xFFFFFFFFu ? mass_ge(p + 1) : 0.0);
            const int ties = count_ge(p) - (p < 0xFFFFFFFFu ? count_ge(p + 1) : 0);
            const double mp = fmax(static_cast<double>(order_bits_to_float(p)), 0.0);
            r = 1;
            while (r < ties && hi + static_cast<double>(r) * mp < target) ++r;
        }
    }
    if (keep >= 0) {
        if (keep == 0) {
            p = 0xFFFFFFFFu;
            r = 0;
        } else if (keep >= n_free) {
            p = 0;
            r = 0;
        } else {
            p = kth_bits(keep);
            r = keep - (p < 0xFFFFFFFFu ? count_ge(p + 1) : 0);
        }
    }
    // flags: 1 kept, 2 at the boundary (resolved below in ascending j)
#pragma unroll
    for (int e = 0; e < EW; ++e) {
        const int j = lane + 64 * e;
        if (vb[e] > p)
            flag[j] = 1;
        else if (vb[e] == p && vb[e] != 0)
            flag[j] = 2;
    }
    wave_sync_lds();
    uint8_t f[EW];
    int nt = 0;
#pragma unroll
    for (int e = 0; e < EW; ++e) {
        f[e] = flag[EW * lane + e];
        nt += f[e] == 2;
    }
    int tr = wave_inclusive_scan(nt, lane) - nt;   // boundary keys before this lane
    int cnt = 0;
#pragma unroll
    for (int e = 0; e < EW; ++e) {
        if (f[e] == 2) f[e] = tr++ < r ? 1 : 0;
        cnt += f[e];
    }

    // compaction in ascending j
    const int incl_c = wave_inclusive_scan(cnt, lane);
    int pos = incl_c - cnt;
    const int total = __shfl(incl_c, 63);
    const size_t orow = (size_t)bh * ldn + i;     // row of the [BH, ldn, ldn] lists
    int32_t* out = kv_idx + orow * ldn;
#pragma unroll
    for (int e = 0; e < EW; ++e) {
        const int j = EW * lane + e;
        if (f[e]) out[pos++] = j;
    }
    for (int j = n + lane; j < ldn; j += 64) out[total + (j - n)] = j;
    if (lane == 0) kv_cnt[orow] = total + (ldn - n);
}

inline unsigned cdiv(long a, long b) { return static_cast<unsigned>((a + b - 1) / b); }

}  // namespace

// ---------------------------------------------------------------------------
// a5, pattern form (Section 5.3): per head, the K largest of the 3n - 1
// predicted pattern intensities (diagonals delta = -(n-1)..n-1 at index
// delta + n - 1, then columns j at 2n - 1 + j), keys at float32 precision,
// ties by pattern index.  The 64-bit key (order_bits(value) << 32 | ~index)
// is unique, so the K-th largest key is found exactly by an 8-pass radix
// select over 8-bit digits; a pattern is chosen iff its key reaches it.
// Then per row, block (i, j) is kept iff its diagonal or its column is
// chosen or it is forced; the kept blocks are compacted in ascending j.
// ---------------------------------------------------------------------------
__device__ inline uint64_t pattern_key(const double* v, int p) {
    return (static_cast<uint64_t>(order_bits(static_cast<float>(v[p]))) << 32) |
           static_cast<uint64_t>(0xFFFFFFFFu - static_cast<uint32_t>(p));
}

__global__ __launch_bounds__(kThreads) void pattern_rank_kernel(const double* __restrict__ pred,
                                                                 uint8_t* __restrict__ chosen,
                                                                 int n, int K) {
    __shared__ uint32_t hist[256];
    __shared__ uint64_t s_prefix;
    __shared__ int s_need;
    const int P = 3 * n - 1;
    const int bh = blockIdx.x, t = threadIdx.x;
    const double* v = pred + (size_t)bh * P;
    if (t == 0) {
        s_prefix = 0;
        s_need = K;
    }
    for (int pass = 0; pass < 8; ++pass) {
        const int shift = 56 - 8 * pass;
        const uint64_t hi_mask = pass == 0 ? 0ull : (~0ull << (shift + 8));
        hist[t] = 0;      // kThreads == 256 bins
        __syncthreads();
        const uint64_t prefix = s_prefix;
        for (int q = t; q < P; q += kThreads) {
            const uint64_t key = pattern_key(v, q);
            if ((key & hi_mask) == prefix) atomicAdd(&hist[(key >> shift) & 255u], 1u);
        }
        __syncthreads();
        if (t == 0) {
            int need = s_need;
            uint32_t cum = 0;
            for (int dgt = 255; dgt >= 0; --dgt) {
                if (cum + hist[dgt] >= (uint32_t)need) {
                    s_prefix = prefix | (static_cast<uint64_t>(dgt) << shift);
                    s_need = need - (int)cum;
                    break;
                }
                cum += hist[dgt];
            }
        }
        __syncthreads();
    }
    const uint64_t kth = s_prefix;    // the K-th largest key (keys are unique)
    for (int q = t; q < P; q += kThreads) chosen[(size_t)bh * P + q] = pattern_key(v, q) >= kth ? 1 : 0;
}

__global__ __launch_bounds__(kThreads) void pattern_rows_kernel(
    const uint8_t* __restrict__ chosen, const int32_t* __restrict__ gate,
    const int* __restrict__ row_lo, const int* __restrict__ row_hi, int32_t* __restrict__ kv_idx,
    int32_t* __restrict__ kv_cnt, int n, int ldn, int tb0) {
    __shared__ int wtot[kThreads / 64];
    constexpr int JPT = kMaxBlocks / kThreads;
    const int row = blockIdx.x;
    const int bh = row / n, i = row % n;
    const uint8_t* ch = chosen + (size_t)bh * (3 * n - 1);
    const bool g = gate[bh] != 0;
    const int flo = row_lo[i], fhi = row_hi[i];
    const int t = threadIdx.x, lane = t & 63, w = t >> 6;
    bool keep[JPT];
    int mine = 0;
#pragma unroll
    for (int e = 0; e < JPT; ++e) {
        const int j = t * JPT + e;
        keep[e] = j < n && (ch[j - i + n - 1] || ch[2 * n - 1 + j] || (g && j >= flo && j <= fhi) ||
                            j == tb0);
        mine += keep[e] ? 1 : 0;
    }
    int incl = mine;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const int y = __shfl_up(incl, off);
        if (lane >= off) incl += y;
    }
    if (lane == 63) wtot[w] = incl;
    __syncthreads();
    int pos = incl - mine, total = 0;
#pragma unroll
    for (int ww = 0; ww < kThreads / 64; ++ww) {
        pos += ww < w ? wtot[ww] : 0;
        total += wtot[ww];
    }
    const size_t orow = (size_t)bh * ldn + i;     // row of the [BH, ldn, ldn] lists
    int32_t* out = kv_idx + orow * ldn;
#pragma unroll
    for (int e = 0; e < JPT; ++e)
        if (keep[e]) out[pos++] = t * JPT + e;
    // text blocks after the video blocks: kept in every row
    for (int j = n + t; j < ldn; j += kThreads) out[total + (j - n)] = j;
    if (t == 0) kv_cnt[orow] = total + (ldn - n);
}

// Token-type-aware masking: the rows of the blocks holding text tokens
// (tb0 .. ldn-1) keep every block.  Grid (ldn - tb0, BH).
__global__ __launch_bounds__(kThreads) void text_rows_kernel(int32_t* __restrict__ kv_idx,
                                                             int32_t* __restrict__ kv_cnt, int ldn,
                                                             int tb0) {
    const size_t orow = (size_t)blockIdx.y * ldn + tb0 + blockIdx.x;
    int32_t* out = kv_idx + orow * ldn;
    for (int j = threadIdx.x; j < ldn; j += kThreads) out[j] = j;
    if (threadIdx.x == 0) kv_cnt[orow] = ldn;
}

hipError_t launch_pool(const uint16_t* q, const uint16_t* k, double* qbar, double* kbar,
                       int BH, int L, int L_stride, int d, int bs, int n, hipStream_t s) {
    const dim3 grid(n, BH, 2);
    if (d == 128 && bs == 128)
        hipLaunchKernelGGL((pool_kernel<128, 128>), grid, dim3(kThreads), 0, s, q, k, qbar, kbar, L, L_stride, n);
    else if (d == 128)
        hipLaunchKernelGGL((pool_kernel<128, 64>), grid, dim3(kThreads), 0, s, q, k, qbar, kbar, L, L_stride, n);
    else if (bs == 128)
        hipLaunchKernelGGL((pool_kernel<64, 128>), grid, dim3(kThreads), 0, s, q, k, qbar, kbar, L, L_stride, n);
    else
        hipLaunchKernelGGL((pool_kernel<64, 64>), grid, dim3(kThreads), 0, s, q, k, qbar, kbar, L, L_stride, n);
    return hipGetLastError();
}

hipError_t launch_block_mass(const double* qbar, const double* kbar, double* G, int BH,
                             int L, int d, int bs, int n, double scale, hipStream_t s) {
    const dim3 grid(cdiv(n, 128), cdiv(n, 128), BH);
    if (d == 128)
        hipLaunchKernelGGL(logits_kernel<128>, grid, dim3(kThreads), 0, s, qbar, kbar, G, n, scale);
    else
        hipLaunchKernelGGL(logits_kernel<64>, grid, dim3(kThreads), 0, s, qbar, kbar, G, n, scale);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(mass_softmax_kernel, dim3((unsigned)BH * n), dim3(kThreads), 0, s, G, L,
                       bs, n);
    return hipGetLastError();
}

hipError_t launch_rhs(const double* G, const int* reg, double* r, double* part, int BH, int n, int F,
                      hipStream_t s) {
    hipLaunchKernelGGL(rhs_kernel, dim3(cdiv(3 * n - 1, kThreads), kRhsChunks, BH), dim3(kThreads), 0, s, G, part,
                       BH, n);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(rhs_sum_kernel, dim3(cdiv(3 * n - 1, kThreads), BH), dim3(kThreads), 0, s, part, r, BH, n, F);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(rhs_frame_kernel, dim3(F, BH), dim3(kThreads), 0, s, G, reg, r, n, F);
    return hipGetLastError();
}

hipError_t launch_solve(const double* r, const int* reg, const double* Sinv, double* bU,
                        double* u, double* X, int BH, int n, int F, hipStream_t s) {
    const int q = n - 1 + F;
    hipLaunchKernelGGL(solve_pre_kernel, dim3(cdiv(q, kThreads), BH), dim3(kThreads),
                       (size_t)(2 * n - 1) * sizeof(double), s, r, reg, bU, n, F);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(solve_gemv_kernel, dim3(cdiv(q, 64), kSolveSplit), dim3(kThreads), 0, s, Sinv, bU,
                       u, q, BH);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(solve_post_kernel, dim3(BH), dim3(kThreads), (size_t)q * sizeof(double) + (size_t)F * sizeof(int),
                       s, r, u, reg, X, n, F, BH);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(solve_gauge_kernel, dim3(BH), dim3(kThreads), 0, s, X, n, F);
    return hipGetLastError();
}

hipError_t launch_gate(const double* Xa, const double* Xb, int32_t* gate, int BH, int n,
                       int F, double tau_e, hipStream_t s) {
    hipLaunchKernelGGL(gate_kernel, dim3(cdiv(BH, 64)), dim3(64), 0, s, Xa, Xb, gate, BH, n, F,
                       tau_e);
    return hipGetLastError();
}

hipError_t launch_extrapolate(const double* X1, const double* X2, double w, double* pred,
                              int BH, int n, int F, hipStream_t s) {
    hipLaunchKernelGGL(extrapolate_kernel, dim3(cdiv(3 * n - 1, kThreads), BH), dim3(kThreads), 0,
                       s, X1, X2, w, pred, n, F);
    return hipGetLastError();
}

hipError_t launch_text_rows(int32_t* kv_idx, int32_t* kv_cnt, int BH, int ldn, int tb0, hipStream_t s) {
    if (tb0 >= ldn) return hipSuccess;
    hipLaunchKernelGGL(text_rows_kernel, dim3((unsigned)(ldn - tb0), (unsigned)BH), dim3(kThreads), 0, s,
                       kv_idx, kv_cnt, ldn, tb0);
    return hipGetLastError();
}

hipError_t launch_select(const double* pred, const int32_t* gate, const int* row_lo,
                         const int* row_hi, int mode, int k, double tau, int32_t* kv_idx,
                         int32_t* kv_cnt, int BH, int n, int ldn, int tb0, hipStream_t s) {
    int npad_w = 64;
    while (npad_w < n) npad_w <<= 1;
    if (npad_w <= 1024) {   // one wave per row
        const int rows = BH * n;
        auto gow = [&](auto kern) {
            hipLaunchKernelGGL(kern, dim3(cdiv(rows, kThreads / 64)), dim3(kThreads), 0, s, pred, gate, row_lo,
                               row_hi, mode, k, tau, kv_idx, kv_cnt, n, ldn, tb0, rows);
            return hipGetLastError();
        };
        hipError_t e;
        switch (npad_w / 64) {
            case 1: e = gow(select_wave_kernel<1>); break;
            case 2: e = gow(select_wave_kernel<2>); break;
            case 4: e = gow(select_wave_kernel<4>); break;
            case 8: e = gow(select_wave_kernel<8>); break;
            default: e = gow(select_wave_kernel<16>); break;
        }
        if (e != hipSuccess) return e;
        return launch_text_rows(kv_idx, kv_cnt, BH, ldn, tb0, s);
    }
    int npad = kThreads;
    while (npad < n) npad <<= 1;
    const size_t lds = (size_t)npad * sizeof(int);
    auto go = [&](auto kern) {
        hipLaunchKernelGGL(kern, dim3((unsigned)BH * n), dim3(kThreads), lds, s, pred, gate, row_lo, row_hi,
                           mode, k, tau, kv_idx, kv_cnt, n, ldn, tb0);
        return hipGetLastError();
    };
    hipError_t e;
    switch (npad / kThreads) {
        case 1: e = go(select_kernel<1>); break;
        case 2: e = go(select_kernel<2>); break;
        case 4: e = go(select_kernel<4>); break;
        case 8: e = go(select_kernel<8>); break;
        default: e = go(select_kernel<16>); break;
    }
    if (e != hipSuccess) return e;
    return launch_text_rows(kv_idx, kv_cnt, BH, ldn, tb0, s);
}

hipError_t launch_select_patterns(const double* pred, const int32_t* gate, const int* row_lo,
                                  const int* row_hi, int K, uint8_t* chosen, int32_t* kv_idx,
                                  int32_t* kv_cnt, int BH, int n, int ldn, int tb0, hipStream_t s) {
    hipLaunchKernelGGL(pattern_rank_kernel, dim3((unsigned)BH), dim3(kThreads), 0, s, pred, chosen, n, K);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(pattern_rows_kernel, dim3((unsigned)BH * n), dim3(kThreads), 0, s, chosen, gate,
                       row_lo, row_hi, kv_idx, kv_cnt, n, ldn, tb0);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_text_rows(kv_idx, kv_cnt, BH, ldn, tb0, s);
}

}  // namespace moddit
