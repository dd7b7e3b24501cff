// Internal launch interface of the MOD-DiT gfx950 kernels.  Every launcher
// enqueues on `s` and returns the launch status; shapes are validated by the
// C ABI layer before any launcher is called.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

namespace moddit {

constexpr int kMaxBlocks = 4096;     // largest n (selection keeps a row in LDS)
constexpr int kSolveSplit = 16;     // k-chunks of the Schur-complement product (fixed: deterministic sum)
constexpr int kRhsChunks = 4;       // row ranges of the right-hand side sums (fixed: deterministic sum)

// a1: block means of Q and K, fp64 [BH, n, d], over the first L tokens of
// each head (L_stride tokens apart).
hipError_t launch_pool(const uint16_t* q, const uint16_t* k, double* qbar, double* kbar,
                       int BH, int L, int L_stride, int d, int bs, int n, hipStream_t s);

// a2: pooled block-mass statistic G [BH, n, n] fp64 (row-stochastic).
hipError_t launch_block_mass(const double* qbar, const double* kbar, double* G, int BH,
                             int L, int d, int bs, int n, double scale, hipStream_t s);

// a3: right-hand side M^T vec(G) [BH, p] and the structured minimum-norm
// solve into X [BH, p].  reg: [F][2] inclusive block ranges; Sinv: inverse
// of the Schur complement [q, q], q = n - 1 + F; bU: scratch [BH, q];
// u: scratch [kSolveSplit, BH, q] (partial products per k-chunk).
// part: scratch of kRhsChunks * BH * (3n - 1) doubles (the row ranges' sums).
hipError_t launch_rhs(const double* G, const int* reg, double* r, double* part, int BH, int n, int F,
                      hipStream_t s);
hipError_t launch_solve(const double* r, const int* reg, const double* Sinv, double* bU,
                        double* u, double* X, int BH, int n, int F, hipStream_t s);

// Block-diagonal gate per head from one or two anchors (Xb may equal Xa).
hipError_t launch_gate(const double* Xa, const double* Xb, int32_t* gate, int BH, int n,
                       int F, double tau_e, hipStream_t s);

// a4: pred [BH, 3n-1] = x2 + (x2 - x1) * w over the c and d parts.
hipError_t launch_extrapolate(const double* X1, const double* X2, double w, double* pred,
                              int BH, int n, int F, hipStream_t s);

// a5: per-row selection into compacted lists.  row_lo/row_hi: union of the
// frame regions holding block i; mode 0 = TOPK (k), 1 = MASS (tau).
// n: video blocks; ldn >= n: blocks of the whole sequence (lists
// [BH, ldn, ldn]); tb0: first text block (ldn when there is no text).  The
// text blocks are kept in every row and the text rows keep every block.
hipError_t launch_select(const double* pred, const int32_t* gate, const int* row_lo,
                         const int* row_hi, int mode, int k, double tau, int32_t* kv_idx,
                         int32_t* kv_cnt, int BH, int n, int ldn, int tb0, hipStream_t s);

// a5, pattern form: the K largest pattern intensities per head (chosen
// [BH, 3n-1] bytes, scratch), then per-row lists of the blocks a chosen
// diagonal or column covers, plus the forced blocks.
hipError_t launch_select_patterns(const double* pred, const int32_t* gate, const int* row_lo,
                                  const int* row_hi, int K, uint8_t* chosen, int32_t* kv_idx,
                                  int32_t* kv_cnt, int BH, int n, int ldn, int tb0, hipStream_t s);

// a6: block-sparse attention forward.  ws: device workspace of ws_bytes
// bytes, at least attn_plan_bytes(BH, n, 0) (the work plan, rewritten every
// call); attn_workspace_bytes(BH, n, d, bs) also holds the partial results
// of the split-KV path (split pairs need ws_bytes to hold >= 2 slots).
size_t attn_plan_bytes(int BH, int n, int S);
size_t attn_workspace_bytes(int BH, int n, int d, int bs);
int attn_slots_for(int BH, int n, int d, int bs, size_t ws_bytes);
hipError_t launch_attn_fwd(const uint16_t* q, const uint16_t* k, const uint16_t* v,
                           const int32_t* kv_idx, const int32_t* kv_cnt, float scale,
                           uint16_t* o, float* lse, int BH, int L, int d, int bs, int n,
                           void* ws, size_t ws_bytes, hipStream_t s);

// The attention's work plan in a library-owned device array of
// kNoAllocScratchBytes per device (for callers that cannot allocate):
// the current device's address of that array, resolved on first use.
constexpr size_t kNoAllocScratchBytes = size_t(2) << 20;
hipError_t noalloc_scratch(void** out);

// Eq. 2 statistic of a computed attention map: stat[bh][i][j] = fraction of
// the probabilities of listed block (i, j) that reach exp(log_eta), with the
// row LSE of the attention forward over the same lists; unlisted blocks keep
// their value.  Lists over the n blocks of the sequence; stat [BH, nv, nv]
// over its first nv (video) blocks.
hipError_t launch_stat_count(const uint16_t* q, const uint16_t* k, const int32_t* kv_idx,
                             const int32_t* kv_cnt, const float* lse, float scale, float log_eta,
                             double* stat, int BH, int L, int d, int bs, int n, int nv, hipStream_t s);

}  // namespace moddit
