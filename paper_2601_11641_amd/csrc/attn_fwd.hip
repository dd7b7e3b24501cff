// Block-sparse attention forward for gfx950 (Eq. 1 with a block mask).
//
// One work item per (head, pair of query blocks 2p, 2p+1), processed by a
// persistent work-group (one per compute unit, items fetched from a work
// plan written before the launch) with 2 * BS/32 waves in two groups: group g
// owns query block 2p+g, wave qw of a group owns 32 of its query rows.  The
// union of the two kv lists is walked in two parts.  First the blocks in
// both lists: every K/V tile brought into LDS serves both groups.  Then the
// blocks in one list only, both groups at once: group 0 walks those of
// block 2p while group 1 walks those of block 2p+1, each with its own
// buffers, so neither group waits through a tile the other one alone needs.
// Every wave runs an online softmax over whole tiles, half a tile (a "unit")
// at a time; the order of the tiles does not change the result beyond
// rounding.
//
// Per unit a wave has two phases:
//   M  S^T (kv x q) = K . Q^T with v_mfma_f32_32x32x16_bf16 (a lane owns one
//      query column, so the row max and the rescale are per-lane scalars),
//      and the product of the previous unit, O^T (d x q) += V^T . P^T, whose
//      V^T operand comes from the row-major V tile through
//      ds_read_b64_tr_b16 (transposing LDS reads);
//   X  the softmax step: P = exp2(S * scale*log2e - m) in fp32 with the
//      running max m kept, accepted when no lane's probabilities of the unit
//      sum past 2^8; otherwise (rarely) the unit's max is taken, m moves up
//      to it and O, l are rescaled.  P is rounded to bf16 as the B operand of
//      the next product without moving between lanes.
// Waves of the two groups share every SIMD, and group 1 runs one phase behind
// group 0 with a work-group barrier after every phase: on each SIMD one wave's
// matrix products overlap the other wave's softmax.
//
// K and V tiles (BS x D bf16, row-major, 16-byte chunks XOR-swizzled per row)
// are copied straight into LDS (global_load_lds_dwordx4) during the X phases:
// in the shared part two buffers each, group 0 copying K and group 1 V one
// tile ahead; in the exclusive part one K and one V buffer per group, which
// copies its own tiles half a tile ahead.
#include "moddit_internal.h"

#include <algorithm>
#include <atomic>
#include <mutex>
#include <type_traits>

namespace moddit {
namespace {

typedef __bf16 bf16x8 __attribute__((__vector_size__(8 * sizeof(__bf16))));
typedef short s16x4 __attribute__((__vector_size__(4 * sizeof(short))));
typedef short s16x8 __attribute__((__vector_size__(8 * sizeof(short))));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4_t;

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kSumLimit = 256.0f;    // fast-path bound on a lane's probability sum per unit
constexpr int kXcds = 8;               // accelerator complex dies of an MI355X

// max(x, x of lane l ^ 32): with x in both operands, v_permlane32_swap
// returns x[l mod 32] and x[l mod 32 + 32] to lane l, i.e. its own value and
// its partner's.
__device__ __forceinline__ float max_across_halves(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                    false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// Direct-to-LDS copy of 16 bytes per lane: lane l writes LDS bytes
// [lds + 16 l, +16) with the 16 bytes at sbase + voff (sbase wave-uniform,
// voff the lane's byte offset).  Written as inline assembly so that the
// compiler's wait-count bookkeeping does not treat the copy as a pending LDS
// access (it would otherwise turn every later partial LDS wait into a full
// one); its completion is tracked by vmcnt alone and waited for explicitly
// before the barrier that publishes the tile.  M0 carries the LDS address;
// nothing else in this kernel uses M0.
__device__ __forceinline__ void lds_copy16(const void* sbase, uint32_t voff, const char* lds) {
    const uint32_t m0 = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) char*)lds;
    asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
                 :: "v"(voff), "s"(sbase), "s"(m0) : "memory");
}

// XOR pattern applied to the 16-byte chunk index of a tile row.  The LDS
// serves 256 bytes (64 four-byte banks) per cycle: 16 lanes of a 16-byte
// read, 32 lanes of an 8-byte read.  The MFMA operand loads (16 bytes per
// lane) read one chunk column of 16 aligned consecutive rows per cycle, so
// the pattern must be a permutation over any 16 such rows.  The transposing
// loads (8 bytes per lane) read, per 32 lanes, the same four chunks (64
// bytes) of 4 aligned consecutive rows, so over any such 4 rows the pattern
// must differ in bits 2..3 (the 64-byte quarter of the row).  At D = 128,
// swz(r) = (r&3)<<2 | (r>>2)&3 meets both.  At D = 64 a row (8 chunks)
// covers half the banks and rows of either parity the other half, so the
// conditions hold separately for the even and the odd rows:
// swz(r) = ((r>>1)&1)<<2 | (r>>2)&3.
template <int D>
__device__ __forceinline__ int swz(int row) {
    if constexpr (D == 128)
        return ((row & 3) << 2) | ((row >> 2) & 3);
    else
        return (((row >> 1) & 1) << 2) | ((row >> 2) & 3);
}

// A group's direct-to-LDS copies of one BS x D tile (NW waves, IPW 1-KB
// copies each).  Copy `ins` fills LDS bytes [ins*1024, +1024): lane l writes
// the 16-byte chunk at ins*1024 + 16*l, i.e. row ins*RPI + l/LPR, physical
// chunk l % LPR, which holds logical chunk (l % LPR) ^ swz(row).  The
// per-lane source offset only depends on ins mod 4 (D = 128) or ins mod 2
// (D = 64); it is precomputed in voff.  Rows past the end of the sequence
// (short tail tile) re-read the last valid row: their scores are masked and
// their probabilities are zero.
template <int D, int BS, int NW>
struct TileCopy {
    static constexpr int ROWB = 2 * D;            // bytes per row
    static constexpr int LPR = ROWB / 16;         // lanes per row
    static constexpr int RPI = 64 / LPR;          // rows per 1-KB copy
    static constexpr int IPW = BS * ROWB / 1024 / NW;
    static constexpr int NV = D == 128 ? 4 : 2;
    uint32_t voff[NV];                             // byte offsets, lane part

    __device__ __forceinline__ explicit TileCopy(int lane) {
#pragma unroll
        for (int a = 0; a < NV; ++a) {
            const int row = a * RPI + lane / LPR;  // row mod 16 (D=128) / mod 8 (D=64)
            voff[a] = (uint32_t)((lane / LPR) * ROWB + (((lane % LPR) ^ swz<D>(row)) << 4));
        }
    }

    // Copy ii of wave w (within the group) of a full tile whose first row
    // starts at byte address gt.
    __device__ __forceinline__ void issue_one(const char* gt, int ii, char* tile, int w) const {
        const int ins = w * IPW + ii;
        lds_copy16(gt + (size_t)ins * 1024, voff[ii % NV], tile + ins * 1024);
    }

    // All copies of wave w of a short tile (kvalid < BS valid rows starting
    // at row k0 of the head whose first element is g).
    __device__ __forceinline__ void issue_tail(const uint16_t* __restrict__ g, int k0, int kvalid,
                                               char* tile, int w, int lane) const {
#pragma unroll
        for (int ii = 0; ii < IPW; ++ii) {
            const int ins = w * IPW + ii;
            const int row = ins * RPI + lane / LPR;
            const int chunk = (lane % LPR) ^ swz<D>(row);
            const uint32_t off = (uint32_t)((k0 + min(row, kvalid - 1)) * ROWB + chunk * 16);
            lds_copy16(g, off, tile + ins * 1024);
        }
    }

    // Start copying tile j (rows j*BS ..) of head g into `tile`: a full tile
    // is returned as a source address for issue_one, a short one is issued
    // at once and nullptr is returned.
    __device__ __forceinline__ const char* start(const uint16_t* __restrict__ g, int j, int L, char* tile,
                                                 int w, int lane) const {
        const int kvalid = min(BS, L - j * BS);
        if (kvalid == BS) return reinterpret_cast<const char*>(g + (size_t)j * BS * D);
        issue_tail(g, j * BS, kvalid, tile, w, lane);
        return nullptr;
    }

    __device__ __forceinline__ void issue_all(const uint16_t* __restrict__ g, int j, int L, char* tile, int w,
                                              int lane) const {
        const char* gt = start(g, j, L, tile, w, lane);
        if (gt != nullptr) {
#pragma unroll
            for (int ii = 0; ii < IPW; ++ii) issue_one(gt, ii, tile, w);
        }
    }

    // Half tiles (rows [hh*BS/2, (hh+1)*BS/2)): IPH copies per wave, the
    // same LDS layout as the full tile.
    static constexpr int IPH = IPW / 2;
    static constexpr int CPH = IPH * NW;          // copies per half tile

    __device__ __forceinline__ void issue_half_one(const char* gt, int hh, int ii, char* tile, int w) const {
        static_assert(IPH % NV == 0, "a wave's first copy of a half must start a swizzle period");
        const int ins = hh * CPH + w * IPH + ii;
        lds_copy16(gt + (size_t)ins * 1024, voff[ii % NV], tile + ins * 1024);
    }

    // Start copying half hh of tile j: a full tile is returned as a source
    // address for issue_half_one, a short one is issued at once (nullptr).
    __device__ __forceinline__ const char* start_half(const uint16_t* __restrict__ g, int j, int L, char* tile,
                                                      int hh, int w, int lane) const {
        const int kvalid = min(BS, L - j * BS);
        if (kvalid == BS) return reinterpret_cast<const char*>(g + (size_t)j * BS * D);
#pragma unroll
        for (int ii = 0; ii < IPH; ++ii) {
            const int ins = hh * CPH + w * IPH + ii;
            const int row = ins * RPI + lane / LPR;
            const int chunk = (lane % LPR) ^ swz<D>(row);
            const uint32_t off = (uint32_t)((j * BS + min(row, kvalid - 1)) * ROWB + chunk * 16);
            lds_copy16(g, off, tile + ins * 1024);
        }
        return nullptr;
    }

    __device__ __forceinline__ void issue_half(const uint16_t* __restrict__ g, int j, int L, char* tile, int hh,
                                               int w, int lane) const {
        const char* gt = start_half(g, j, L, tile, hh, w, lane);
        if (gt != nullptr) {
#pragma unroll
            for (int ii = 0; ii < IPH; ++ii) issue_half_one(gt, hh, ii, tile, w);
        }
    }
};

// s_waitcnt vmcnt(N): at most N vector memory operations of the wave still
// outstanding (they complete in issue order).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// f(integral_constant<int, i>) for i = 0 .. N-1, unrolled at compile time.
template <class F, int... I>
__device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, I...>) {
    (f(std::integral_constant<int, I>{}), ...);
}
template <int N, class F>
__device__ __forceinline__ void static_for(F&& f) {
    static_for_impl(f, std::make_integer_sequence<int, N>{});
}

// ---------------------------------------------------------------------------
// Work plan.  The per-pair work (about the two rows' list lengths) varies
// along the sequence and across heads, so a fixed pair -> XCD map leaves
// some XCDs idle at the end.  One small kernel (one work-group per XCD, each
// computing the shared quantities itself) writes a plan into the workspace
// before every attention launch:
//   costs  the cost 4 + cnt(2p) + cnt(2p+1) of every pair p of every head;
//          per head, eight contiguous pair ranges of about equal cost (pair
//          p goes to range floor(8 * midpoint(p) / head total)), one per XCD:
//          neighbouring rows share K/V blocks, so an XCD's L2 serves its
//          range, and all XCDs work through the same heads at once;
//   split  a pair whose cost exceeds half of the average per-CU load
//          W / (compute units) is split into C chunks of its walk (the walk
//          of a pair has max(cnt(2p), cnt(2p+1)) steps: the blocks of both
//          lists, then the one-list blocks of both rows side by side), each
//          of about an eighth of that load and at least kMinChunkSteps
//          steps; the chunks become separate items writing partial results
//          (fp32 O / l and LSE per row) into workspace slots, merged after
//          the launch in chunk order.  If the slots do not suffice, the
//          chunk length doubles until they do (or nothing is split);
//   lists  per XCD, the items of its ranges in head-major order (a chunk
//          item is the slot number with bit 30 set), its length, start and
//          a zeroed fetch counter; each list is then bucket-sorted by
//          decreasing cost (lists longer than kPlanSortMax keep the head
//          order), so long items start early instead of ending the launch
//          late.
// Every work-group computes the same split decision and slot numbering from
// the same counts, so the plan is deterministic; only the order of equal-
// cost items within a bucket varies, which affects timing, not results.
// The attention work-groups are persistent (one per CU): a work-group
// fetches the next item of its XCD's list with an atomic counter and, once
// that list is drained, of the other XCDs' lists, until all are drained.
// Each counter has a 128-byte line of its own, so the XCDs' atomics do not
// queue on one line.
// ---------------------------------------------------------------------------
constexpr int kPlanThreads = 1024;
constexpr int kCtrStride = 32;        // ints between fetch counters (one 128-byte line each)
constexpr int kPlanHdr = 8 * kCtrStride + 32;   // ints: ctr[8] (strided), len[8], start[8], misc[8]
constexpr int kPlanSortMax = 8192;    // longer XCD lists keep the head order
constexpr int kPlanBuckets = 512;
constexpr int kChunkBit = 1 << 30;    // item flag: a chunk of a split pair (slot in the low bits)
constexpr int kMinChunkSteps = 64;    // shortest chunk of a split walk
constexpr int kMaxSplitSlots = 1024;  // partial-result slots a workspace holds at most
constexpr int kPlanCache = 16384;     // pairs whose counts the plan keeps in LDS

// Work-plan layout in the workspace (ints, then the partial-result slots).
struct Plan {
    int* ctr;           // fetch counters, ctr[kCtrStride * x] for XCD x
    int* len;           // [8] items per XCD list
    int* start;         // [8] first item of each XCD list in `items`
    int* misc;          // [0] split pairs, [1] chunk length in steps (0: none)
    long long* headpre; // [8][BH + 1] per work-group: cost before each head's first pair
    int* items;         // [BH * npairs + S]
    int4* chunks;       // [S] chunk items: {pair, first step, end step, 0}
    int4* splits;       // [S] split pairs: {pair, chunks, first slot, 0}
    float* part;        // [S] slots of partial results
    __host__ __device__ static size_t ints(int BH, int npairs, int S) {
        size_t w = (size_t)kPlanHdr + 2 * 8 * ((size_t)BH + 1) + (size_t)BH * npairs + S;
        w = (w + 3) / 4 * 4 + 8 * (size_t)S;
        return (w + 63) / 64 * 64;
    }
    __host__ __device__ Plan(void* ws, int BH, int npairs, int S) {
        int* w = static_cast<int*>(ws);
        ctr = w;
        len = w + 8 * kCtrStride;
        start = len + 8;
        misc = start + 8;
        headpre = reinterpret_cast<long long*>(w + kPlanHdr);
        items = w + kPlanHdr + 2 * 8 * ((size_t)BH + 1);
        size_t o = (size_t)kPlanHdr + 2 * 8 * ((size_t)BH + 1) + (size_t)BH * npairs + S;
        o = (o + 3) / 4 * 4;
        chunks = reinterpret_cast<int4*>(w + o);
        splits = chunks + S;
        part = reinterpret_cast<float*>(w + ints(BH, npairs, S));
    }
};

// Floats per partial-result slot: O / l for the BS x D rows of both query
// blocks of a pair, then their LSE.
__host__ __device__ constexpr size_t slot_floats(int D, int BS) { return 2 * (size_t)BS * D + 2 * (size_t)BS; }

__device__ __forceinline__ int clamp_count(const int32_t* kv_cnt, size_t row, int n) {
    return min(max(kv_cnt[row], 0), n);
}

// Work-group sums and exclusive scans over kPlanThreads threads: a scan
// within each wave by lane shuffles, the waves' totals through buf (at least
// kPlanThreads / 64 entries), two barriers.
template <class T>
__device__ T plan_scan(T v, T* buf, T& total) {
    constexpr int NW = kPlanThreads / 64;
    const int t = threadIdx.x, lane = t & 63, w = t >> 6;
    T incl = v;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const T y = __shfl_up(incl, off);
        if (lane >= off) incl += y;
    }
    if (lane == 63) buf[w] = incl;
    __syncthreads();
    T base = T(0), tot = T(0);
#pragma unroll
    for (int ww = 0; ww < NW; ++ww) {
        const T s = buf[ww];
        base += ww < w ? s : T(0);
        tot += s;
    }
    total = tot;
    __syncthreads();   // buf is free for the next scan
    return base + incl - v;
}

__global__ __launch_bounds__(kPlanThreads) void plan_kernel(const int32_t* __restrict__ kv_cnt, void* ws,
                                                            int BH, int n, int ncu, int S) {
    __shared__ long long scan64[kPlanThreads / 64];
    __shared__ int scan32[kPlanThreads / 64];
    __shared__ int xcnt[kXcds];
    __shared__ uint32_t cache[kPlanCache];   // both counts of a pair, 16 bits each
    const int x = blockIdx.x, t = threadIdx.x;
    const int npairs = (n + 1) / 2;
    const long long P = (long long)BH * npairs;
    const Plan pl(ws, BH, npairs, S);
    long long* hp = pl.headpre + (size_t)x * (BH + 1);
    const long long per = (P + kPlanThreads - 1) / kPlanThreads;
    const long long q0 = min(P, (long long)t * per), q1 = min(P, q0 + per);
    struct Pair { int c0, c1; };
    auto load_counts = [&](long long q) {
        const int bh = (int)(q / npairs), p = (int)(q % npairs);
        const size_t r0 = (size_t)bh * n + 2 * p;
        return Pair{clamp_count(kv_cnt, r0, n), 2 * p + 1 < n ? clamp_count(kv_cnt, r0 + 1, n) : 0};
    };
    // head and pair index of q0, advanced pair by pair in the loops below
    // (no division per pair)
    const int h0 = (int)(q0 / npairs), p0 = (int)(q0 % npairs);
    // every pass reads the counts: from LDS when they fit (loaded once,
    // coalesced), else from the lists' counts in memory
    const bool cached = P <= kPlanCache;
    if (cached) {
        // every thread's loads issued at once (indices clamped to the last
        // pair, so that no load sits behind a branch), then stored
        constexpr int FILL = kPlanCache / kPlanThreads;
        const int Pi = (int)P;
        int c0[FILL], c1[FILL];
#pragma unroll
        for (int u = 0; u < FILL; ++u) {
            const int q = min(t + u * kPlanThreads, Pi - 1);
            const int bh = q / npairs, pp = q - bh * npairs;
            const size_t r0 = (size_t)bh * n + 2 * pp;
            c0[u] = kv_cnt[r0];
            c1[u] = kv_cnt[2 * pp + 1 < n ? r0 + 1 : r0];
        }
#pragma unroll
        for (int u = 0; u < FILL; ++u) {
            const int q = t + u * kPlanThreads;
            const int pp = q % npairs;
            const int a = min(max(c0[u], 0), n), b = 2 * pp + 1 < n ? min(max(c1[u], 0), n) : 0;
            if (q < Pi) cache[q] = (uint32_t)a | ((uint32_t)b << 16);
        }
        __syncthreads();
    }
    auto counts = [&](long long q) {
        if (cached) {
            const uint32_t v = cache[q];
            return Pair{(int)(v & 0xFFFF), (int)(v >> 16)};
        }
        return load_counts(q);
    };
    // cost before every pair (global order) and before every head
    long long mine = 0;
    for (long long q = q0; q < q1; ++q) {
        const Pair c = counts(q);
        mine += 4 + c.c0 + c.c1;
    }
    long long W = 0;
    const long long pre = plan_scan<long long>(mine, scan64, W);
    {
        long long run = pre;
        int h = h0, pp = p0;
        for (long long q = q0; q < q1; ++q) {
            const Pair c = counts(q);
            if (pp == 0) hp[h] = run;
            run += 4 + c.c0 + c.c1;
            if (++pp == npairs) { pp = 0; ++h; }
        }
        if (t == 0) hp[BH] = W;
    }
    __syncthreads();   // the head prefixes (this work-group's own copy) are visible
    // split policy: chunks of cs steps for pairs costing more than half the
    // per-CU load, cs doubled until the chunks fit the slots
    const double A = (double)W / (double)max(ncu, 1);
    long long cs = 0;
    auto nchunks = [&](const Pair& c, long long csteps) -> long long {
        const long long cost = 4 + c.c0 + c.c1;
        const long long steps = max(c.c0, c.c1);
        if (csteps <= 0 || (double)cost <= 0.5 * A || steps <= csteps) return 1;
        return (steps + csteps - 1) / csteps;
    };
    if (S >= 2) {
        cs = max((long long)kMinChunkSteps, (long long)(A / 8.0));
        for (;;) {
            long long need = 0;
            for (long long q = q0; q < q1; ++q) {
                const long long C = nchunks(counts(q), cs);
                if (C > 1) need += C;
            }
            long long tot_need = 0;
            (void)plan_scan<long long>(need, scan64, tot_need);
            if (tot_need <= S) break;
            cs *= 2;
            if (cs > n) { cs = 0; break; }
        }
    }
    // XCD of every pair: its head's cost range (from hb, tot long), by the
    // pair's midpoint, min(7, floor(8 mid2 / (2 tot))) counted by comparisons
    // (a head's cost is at most npairs (4 + 2n) < 2^25, so its midpoints
    // and their multiples of tot stay inside 32 bits)
    auto xcd_of = [&](long long hb, long long tot, long long before, const Pair& c) {
        const int mid4 = 4 * (2 * (int)(before - hb) + 4 + c.c0 + c.c1);
        const int tt = (int)tot;
        int xq = 0;
#pragma unroll
        for (int k = 1; k < kXcds; ++k) xq += mid4 >= k * tt ? 1 : 0;
        return xq;
    };
    // the head prefixes of a thread's current head, read again only when
    // its range crosses into the next head
    struct HeadWalk {
        int h, pp;
        long long hb, tot;
    };
    auto head_start = [&]() {
        HeadWalk hw{h0, p0, 0, 1};
        if (q0 < q1) {
            hw.hb = hp[h0];
            hw.tot = hp[h0 + 1] - hw.hb;
        }
        return hw;
    };
    auto head_next = [&](HeadWalk& hw, long long q) {
        if (++hw.pp == npairs) {
            hw.pp = 0;
            ++hw.h;
            if (q + 1 < q1) {
                hw.hb = hp[hw.h];
                hw.tot = hp[hw.h + 1] - hw.hb;
            }
        }
    };
    int cntx[kXcds] = {};
    long long slots_mine = 0, splits_mine = 0;
    {
        long long run = pre;
        HeadWalk hw = head_start();
        for (long long q = q0; q < q1; ++q) {
            const Pair c = counts(q);
            const int xq = xcd_of(hw.hb, hw.tot, run, c);
            head_next(hw, q);
            const long long C = nchunks(c, cs);
#pragma unroll
            for (int xx = 0; xx < kXcds; ++xx) cntx[xx] += xx == xq ? (int)C : 0;
            if (C > 1) {
                slots_mine += C;
                splits_mine += 1;
            }
            run += 4 + c.c0 + c.c1;
        }
    }
    if (t < kXcds) xcnt[t] = 0;
    __syncthreads();
    for (int xx = 0; xx < kXcds; ++xx)
        if (cntx[xx]) atomicAdd(&xcnt[xx], cntx[xx]);
    __syncthreads();
    int first = 0;
    for (int xx = 0; xx < x; ++xx) first += xcnt[xx];
    const int lenx = xcnt[x];
    long long dummy = 0;
    const long long posx = plan_scan<long long>((long long)cntx[x], scan64, dummy);
    const long long slot0 = plan_scan<long long>(slots_mine, scan64, dummy);
    long long nsplit = 0;
    const long long split0 = plan_scan<long long>(splits_mine, scan64, nsplit);
    // this XCD's items, head-major; the chunks of a split pair described
    {
        long long run = pre, pos = first + posx, slot = slot0, sidx = split0;
        HeadWalk hw = head_start();
        for (long long q = q0; q < q1; ++q) {
            const Pair c = counts(q);
            const int xq = xcd_of(hw.hb, hw.tot, run, c);
            head_next(hw, q);
            const long long C = nchunks(c, cs);
            if (C == 1) {
                if (xq == x) pl.items[pos++] = (int)q;
            } else {
                const long long steps = max(c.c0, c.c1);
                if (xq == x) {
                    pl.splits[sidx] = make_int4((int)q, (int)C, (int)slot, 0);
                    for (long long cc = 0; cc < C; ++cc) {
                        pl.chunks[slot + cc] = make_int4((int)q, (int)(cc * steps / C), (int)((cc + 1) * steps / C), 0);
                        pl.items[pos++] = kChunkBit | (int)(slot + cc);
                    }
                }
                slot += C;
                sidx += 1;
            }
            run += 4 + c.c0 + c.c1;
        }
    }
    if (t == 0) {
        pl.len[x] = lenx;
        pl.start[x] = first;
        pl.ctr[kCtrStride * x] = 0;
        if (x == 0) {
            pl.misc[0] = (int)nsplit;
            pl.misc[1] = (int)cs;
        }
    }
    // Longest items first: a bucket sort of the list by decreasing cost
    // (order within a bucket unspecified; the order only affects timing).
    if (lenx > kPlanSortMax) return;
    __shared__ int vals[kPlanSortMax];
    __shared__ int cursor[kPlanBuckets];
    int shift = 0;
    while (((4 + 2 * n) >> shift) >= kPlanBuckets) ++shift;
    auto bucket = [&](int item) {
        int c;
        if (item & kChunkBit) {
            const int4 ch = pl.chunks[item & (kChunkBit - 1)];
            c = 4 + 2 * (ch.z - ch.y);
        } else {
            const Pair pc = counts(item);
            c = 4 + pc.c0 + pc.c1;
        }
        return (kPlanBuckets - 1) - min(kPlanBuckets - 1, c >> shift);   // descending cost
    };
    for (int bb = t; bb < kPlanBuckets; bb += kPlanThreads) cursor[bb] = 0;
    __syncthreads();   // also: every item (and chunk) of the list has been written
    for (int a = t; a < lenx; a += kPlanThreads) {
        const int it = pl.items[first + a];
        vals[a] = it;
        atomicAdd(&cursor[bucket(it)], 1);
    }
    __syncthreads();
    {   // exclusive scan of the bucket sizes (kPlanBuckets <= kPlanThreads entries)
        static_assert(kPlanBuckets <= kPlanThreads, "one bucket per thread");
        const int c = t < kPlanBuckets ? cursor[t] : 0;
        int all = 0;
        const int ex = plan_scan<int>(c, scan32, all);
        if (t < kPlanBuckets) cursor[t] = ex;
    }
    __syncthreads();
    for (int a = t; a < lenx; a += kPlanThreads) {
        const int it = vals[a];
        pl.items[first + atomicAdd(&cursor[bucket(it)], 1)] = it;
    }
}

// Merge of split pairs: for every row of both query blocks of a split pair,
// LSE = log sum_c exp(lse_c) and O = sum_c exp(lse_c - LSE) O_c over its
// chunks c = 0 .. C-1 in order (rows no chunk reached: O = 0, LSE = -inf).
// Persistent: work-group b takes (split pair, query block) b, b + grid, ...
template <int D, int BS>
__global__ __launch_bounds__(256) void merge_kernel(void* ws, int BH, int n, int S, int L,
                                                    uint16_t* __restrict__ o, float* __restrict__ lse) {
    constexpr int TPR = 256 / BS;          // threads per row
    constexpr int DPT = D / TPR;           // d values per thread
    const int npairs = (n + 1) / 2;
    const Plan pl(ws, BH, npairs, S);
    const int nsplit = pl.misc[0];
    const int t = threadIdx.x, r = t / TPR, d0 = (t % TPR) * DPT;
    for (int m = blockIdx.x; m < 2 * nsplit; m += gridDim.x) {
        const int4 sp = pl.splits[m / 2];
        const int g = m % 2, q = sp.x, C = sp.y;
        const int bh = q / npairs, i = 2 * (q % npairs) + g;
        const int row = i * BS + r;
        if (i >= n || row >= L || q < 0 || bh >= BH || sp.z < 0 || sp.z + C > S) continue;
        float lmax = -INFINITY;
        for (int c = 0; c < C; ++c) {
            const float* sl = pl.part + (size_t)(sp.z + c) * slot_floats(D, BS);
            lmax = fmaxf(lmax, sl[2 * BS * D + g * BS + r]);
        }
        float acc[DPT];
#pragma unroll
        for (int e = 0; e < DPT; ++e) acc[e] = 0.0f;
        float wsum = 0.0f;
        if (lmax > -INFINITY) {
            for (int c = 0; c < C; ++c) {
                const float* sl = pl.part + (size_t)(sp.z + c) * slot_floats(D, BS);
                const float lc = sl[2 * BS * D + g * BS + r];
                const float wgt = lc > -INFINITY ? expf(lc - lmax) : 0.0f;
                wsum += wgt;
                const float4* src = reinterpret_cast<const float4*>(sl + ((size_t)g * BS + r) * D + d0);
#pragma unroll
                for (int e = 0; e < DPT / 4; ++e) {
                    const float4 v4 = src[e];
                    acc[4 * e] += wgt * v4.x;
                    acc[4 * e + 1] += wgt * v4.y;
                    acc[4 * e + 2] += wgt * v4.z;
                    acc[4 * e + 3] += wgt * v4.w;
                }
            }
        }
        const float inv = wsum > 0.0f ? 1.0f / wsum : 0.0f;
        uint16_t* orow = o + ((size_t)bh * L + row) * D + d0;
#pragma unroll
        for (int e = 0; e < DPT / 4; ++e) {
            uint2 pk;
            pk.x = (uint32_t)__builtin_bit_cast(uint16_t, static_cast<__bf16>(acc[4 * e] * inv)) |
                   ((uint32_t)__builtin_bit_cast(uint16_t, static_cast<__bf16>(acc[4 * e + 1] * inv)) << 16);
            pk.y = (uint32_t)__builtin_bit_cast(uint16_t, static_cast<__bf16>(acc[4 * e + 2] * inv)) |
                   ((uint32_t)__builtin_bit_cast(uint16_t, static_cast<__bf16>(acc[4 * e + 3] * inv)) << 16);
            *reinterpret_cast<uint2*>(orow + 4 * e) = pk;
        }
        if (lse != nullptr && t % TPR == 0)
            lse[(size_t)bh * L + row] = wsum > 0.0f ? lmax + logf(wsum) : -INFINITY;
    }
}

// Next item for a work-group on XCD x: its own list first, then the others
// (-1 once every list is drained).  Device-scope atomics: the counters are
// shared by every XCD.
__device__ __forceinline__ int fetch_item(const Plan& pl, int x) {
#pragma unroll 1
    for (int a = 0; a < kXcds; ++a) {
        const int xx = (x + a) % kXcds;
        const int len = pl.len[xx];
        if (len == 0) continue;
        const int k = atomicAdd(&pl.ctr[kCtrStride * xx], 1);
        if (k < len) return pl.items[pl.start[xx] + k];
    }
    return -1;
}

// Membership bytes umask[j] of the kv lists of rows row0 and row0 + 1 (the
// second only if has1) of the [rows, n] lists: bit 0 row0, bit 1 row0 + 1.
// Counts are clamped to [0, n] (a row never reads past its n entries),
// entries outside [0, n) are ignored and a repeated entry counts once.
template <int NT>
__device__ __forceinline__ void mark_rows(const int32_t* __restrict__ kv_idx, const int32_t* __restrict__ kv_cnt,
                                          size_t row0, bool has1, int n, uint8_t* umask, int tid) {
    // the counts and every entry slot of both rows are loaded at once (one
    // memory latency); slot a of a row is used only if a < its count
    constexpr int EPT = kMaxBlocks / NT;
    const int32_t* list0 = kv_idx + row0 * n;
    const int32_t* list1 = list0 + n;
    const int c0 = kv_cnt[row0];
    const int c1 = has1 ? kv_cnt[row0 + 1] : 0;
    int e0[EPT], e1[EPT];
#pragma unroll
    for (int x = 0; x < EPT; ++x) {
        const int a = tid + x * NT;
        e0[x] = a < n ? list0[a] : -1;
        e1[x] = (has1 && a < n) ? list1[a] : -1;
    }
    const int cnt0 = min(max(c0, 0), n);
    const int cnt1 = min(max(c1, 0), n);
    for (int j = tid; j < n; j += NT) umask[j] = 0;
    __syncthreads();
#pragma unroll
    for (int x = 0; x < EPT; ++x) {
        const int j = e0[x];
        if (tid + x * NT < cnt0 && (unsigned)j < (unsigned)n) umask[j] = 1;
    }
    __syncthreads();
#pragma unroll
    for (int x = 0; x < EPT; ++x) {
        const int j = e1[x];
        if (tid + x * NT < cnt1 && (unsigned)j < (unsigned)n) umask[j] |= 2;
    }
    __syncthreads();
}

// Union of the two lists, compacted in ascending j into ulist as
// j | membership << 16.  Every thread of the NT-thread work-group calls it;
// ulist is complete after the caller's next barrier.
template <int NT>
__device__ __forceinline__ int union_of_rows(const int32_t* __restrict__ kv_idx,
                                             const int32_t* __restrict__ kv_cnt, size_t row0, bool has1,
                                             int n, uint8_t* umask, uint32_t* ulist, int* wsum, int tid,
                                             int lane, int w) {
    constexpr int JPT = kMaxBlocks / NT;
    mark_rows<NT>(kv_idx, kv_cnt, row0, has1, n, umask, tid);
    // thread tid compacts entries [tid*JPT, +JPT) after a work-group scan
    int mine = 0;
#pragma unroll
    for (int e = 0; e < JPT; ++e) {
        const int j = tid * JPT + e;
        mine += (j < n && umask[j] != 0) ? 1 : 0;
    }
    int incl = mine;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const int y = __shfl_up(incl, off);
        if (lane >= off) incl += y;
    }
    if (lane == 63) wsum[w] = incl;
    __syncthreads();
    int pos = incl - mine, ucnt = 0;
#pragma unroll
    for (int ww = 0; ww < NT / 64; ++ww) {
        pos += ww < w ? wsum[ww] : 0;
        ucnt += wsum[ww];
    }
#pragma unroll
    for (int e = 0; e < JPT; ++e) {
        const int j = tid * JPT + e;
        if (j < n && umask[j] != 0) ulist[pos++] = (uint32_t)j | ((uint32_t)umask[j] << 16);
    }
    return ucnt;
}

struct UnionParts {
    int ns, na, nb;   // blocks in both lists, in row0's only, in row0 + 1's only
};

// The same union, partitioned: the blocks of both rows first, then those of
// row0 only, then those of row0 + 1 only, each part in ascending j (entries
// j | membership << 16 as above).  wsum holds 2 * NT/64 ints.
template <int NT>
__device__ __forceinline__ UnionParts union_parts(const int32_t* __restrict__ kv_idx,
                                                  const int32_t* __restrict__ kv_cnt, size_t row0, bool has1,
                                                  int n, uint8_t* umask, uint32_t* ulist, int* wsum, int tid,
                                                  int lane, int w) {
    constexpr int JPT = kMaxBlocks / NT;
    mark_rows<NT>(kv_idx, kv_cnt, row0, has1, n, umask, tid);
    // per thread: counts of the three kinds among entries [tid*JPT, +JPT);
    // both and row0-only are packed in 16-bit fields (counts <= kMaxBlocks)
    uint32_t mine01 = 0;
    int mine2 = 0;
#pragma unroll
    for (int e = 0; e < JPT; ++e) {
        const int j = tid * JPT + e;
        const int u = j < n ? umask[j] : 0;
        mine01 += u == 3 ? 1u : (u == 1 ? 0x10000u : 0u);
        mine2 += u == 2 ? 1 : 0;
    }
    uint32_t inc01 = mine01;
    int inc2 = mine2;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const uint32_t y01 = __shfl_up(inc01, off);
        const int y2 = __shfl_up(inc2, off);
        if (lane >= off) {
            inc01 += y01;
            inc2 += y2;
        }
    }
    if (lane == 63) {
        wsum[2 * w] = (int)inc01;
        wsum[2 * w + 1] = inc2;
    }
    __syncthreads();
    uint32_t pos01 = inc01 - mine01, tot01 = 0;
    int pos2 = inc2 - mine2, tot2 = 0;
#pragma unroll
    for (int ww = 0; ww < NT / 64; ++ww) {
        pos01 += ww < w ? (uint32_t)wsum[2 * ww] : 0u;
        pos2 += ww < w ? wsum[2 * ww + 1] : 0;
        tot01 += (uint32_t)wsum[2 * ww];
        tot2 += wsum[2 * ww + 1];
    }
    UnionParts r;
    r.ns = (int)(tot01 & 0xFFFF);
    r.na = (int)(tot01 >> 16);
    r.nb = tot2;
    int p3 = (int)(pos01 & 0xFFFF), p1 = r.ns + (int)(pos01 >> 16), p2 = r.ns + r.na + pos2;
#pragma unroll
    for (int e = 0; e < JPT; ++e) {
        const int j = tid * JPT + e;
        const int u = j < n ? umask[j] : 0;
        const uint32_t ent = (uint32_t)j | ((uint32_t)u << 16);
        if (u == 3) ulist[p3++] = ent;
        if (u == 1) ulist[p1++] = ent;
        if (u == 2) ulist[p2++] = ent;
    }
    return r;
}

template <int D, int BS>
__global__ __launch_bounds__(BS * 4, 1) void attn_fwd_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
    const uint16_t* __restrict__ v, const int32_t* __restrict__ kv_idx,
    const int32_t* __restrict__ kv_cnt, float scale, uint16_t* __restrict__ o,
    float* __restrict__ lse, int L, int n, void* ws, int BH, int S) {
    constexpr int QW = BS / 32;        // waves per group = 32-row query slices of a block
    constexpr int NT = BS * 4;         // threads: two groups of QW waves
    constexpr int KVW = BS / 2;        // kv rows per unit (half a tile)
    constexpr int RT = KVW / 32;       // 32-row kv sub-tiles per unit
    constexpr int DT = D / 32;         // 32-row d tiles of O^T
    constexpr int KK = D / 16;         // 16-deep d chunks of S^T
    constexpr int TILE = BS * D * 2;   // bytes per K or V tile
    constexpr int ROWB = 2 * D;
    constexpr int HALF = KVW * ROWB;   // bytes per half tile
    using Copy = TileCopy<D, BS, QW>;
    constexpr int IPW = Copy::IPW;
    // K and V tile buffers, at fixed distances: the matrix-phase reads name
    // a buffer by a constant offset
    __shared__ __align__(1024) char tiles[4 * TILE];
    char* const kb0 = tiles;
    char* const kb1 = tiles + TILE;
    char* const vb0 = tiles + 2 * TILE;
    char* const vb1 = tiles + 3 * TILE;
    __shared__ uint32_t ulist[kMaxBlocks];     // union of the two lists: j | membership << 16
    __shared__ uint8_t umask[kMaxBlocks];
    __shared__ int wsum[2 * NT / 64];
    __shared__ int item_s[4];          // pair, first step, end step, slot (-1: whole pair)

    // Persistent work-group on XCD blockIdx % 8 (dispatch order): items
    // (head, pair of query blocks 2p, 2p+1, or a chunk of the walk of a
    // split pair) come from the plan.  Every
    // per-item value is derived inside the loop from copies of the thread
    // index and the workspace pointer that the compiler cannot see through,
    // so nothing is hoisted out of the loop to stay live in registers.
    for (;;) {
    int tid = threadIdx.x;
    void* wsi = ws;
    asm volatile("" : "+v"(tid));
    asm volatile("" : "+s"(wsi));
    const int npairs = (n + 1) / 2;
    if (tid == 0) {
        const Plan pl(wsi, BH, npairs, S);
        const int it = fetch_item(pl, blockIdx.x % kXcds);
        int4 desc = make_int4(it, 0, 0x7fffffff, -1);
        if (it >= 0 && (it & kChunkBit)) {
            const int k2 = it & (kChunkBit - 1);
            desc = k2 < S ? pl.chunks[k2] : make_int4(-2, 0, 0, 0);
            desc.w = k2;
        }
        // an item outside the plan's range is skipped (never read past the lists)
        if (desc.x >= 0 && (long long)desc.x >= (long long)BH * npairs) desc.x = -2;
        item_s[0] = desc.x;
        item_s[1] = desc.y;
        item_s[2] = desc.z;
        item_s[3] = desc.w;
    }
    __syncthreads();
    const int item = item_s[0];
    const int step0 = item_s[1], step1 = item_s[2], slot = item_s[3];
    __syncthreads();   // item_s is rewritten only after every wave has read it
    if (item == -1) break;
    if (item < 0) continue;
    const int bh = item / npairs, pr = item % npairs;
    const int lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform
    const int h = lane >> 5, l32 = lane & 31;
    const int qw = w % QW, g = w / QW;          // query slice, group
    const int i = 2 * pr + g;                   // this group's query block (n: none)
    const size_t base = (size_t)bh * L * D;
    const float c2 = scale * kLog2e;
    const int qrow = i * BS + 32 * qw + l32;

    // ---- union of the kv lists of blocks 2p and 2p+1: the ns blocks of
    // both lists, then the na of block 2p's only, then the nb of 2p+1's only ----
    const size_t row0 = (size_t)bh * n + 2 * pr;
    const UnionParts parts = union_parts<NT>(kv_idx, kv_cnt, row0, 2 * pr + 1 < n, n, umask, ulist, wsum, tid, lane, w);
    const int ns = parts.ns, na = parts.na, nb = parts.nb;
    // The first product (before any unit has been computed) multiplies a
    // zero P with the second half of the "previous" V buffer: that half
    // holds zeros rather than whatever the LDS held before.
    for (int e = tid; e < HALF / 16; e += NT) reinterpret_cast<uint4*>(vb1 + HALF)[e] = make_uint4(0, 0, 0, 0);
    __syncthreads();   // publishes the union list and the zeroed half

    // ---- Q slice (B operand of S^T): lane holds Q[qrow][16kk + 8h .. +7] ----
    bf16x8 qreg[KK];
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
        uint4 val = make_uint4(0, 0, 0, 0);
        if (qrow < L)
            val = *reinterpret_cast<const uint4*>(q + base + (size_t)qrow * D + 16 * kk + 8 * h);
        qreg[kk] = __builtin_bit_cast(bf16x8, val);
    }

    f32x16 oacc[DT];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) oacc[dt] = f32x16{};
    f32x16 sacc[RT];
    bf16x8 pb[2 * RT];   // P of the pending product: zero until a unit is computed
#pragma unroll
    for (int c = 0; c < 2 * RT; ++c) pb[c] = bf16x8{};
    float m = -INFINITY, mb = 0.0f, l = 0.0f;   // running max, m * scale * log2(e), row sum

    const Copy copy(lane);
    const uint16_t* kg = k + base;
    const uint16_t* vg = v + base;

    // Per-lane LDS byte offsets within a half tile.  The swizzle of a row
    // only depends on the row mod 16, so the same offsets serve both halves.
    //   K operand (S^T A operand): row 32 rt + l32, chunk 2 kk + h
    const int ka = l32 * ROWB + ((h ^ swz<D>(l32)) << 4);
    //   V^T operand (transposing reads): rows 16 cc + 4h + (lane%16)/4 (+8),
    //   d = 32 dt + 16 ((lane/16)&1) + 4 (lane%4)
    const int s16 = lane & 15, grp = lane >> 4;
    const int tr_row = 4 * h + (s16 >> 2);
    const int c0 = 2 * (grp & 1) + ((s16 & 3) >> 1);
    const int half8 = (s16 & 1) << 3;
    const int va = tr_row * ROWB + ((c0 ^ swz<D>(tr_row)) << 4) + half8;
    const int vb = (tr_row + 8) * ROWB + ((c0 ^ swz<D>(tr_row + 8)) << 4) + half8;
    // LDS addresses of those reads in the current buffers of the shared part
    // (d-chunk kk of K; d-tile dt of V^T, rows 4h.. and 4h+8..), starting in
    // kb0 and vb0.  A read adds its half and row offsets as a constant, which
    // the instruction's offset field holds, so the reads need no address
    // arithmetic; the tile loop moves these values between the two buffers
    // of a kind (one addition each per tile instead of one per read and
    // phase).
    uint32_t kad[KK], vad[2 * DT];
    {
        const uint32_t kb0a = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) char*)kb0;
        const uint32_t vb0a = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) char*)vb0;
#pragma unroll
        for (int kk = 0; kk < KK; ++kk) kad[kk] = kb0a + (uint32_t)(ka ^ (32 * kk));
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
            vad[2 * dt] = vb0a + (uint32_t)(va ^ (64 * dt));
            vad[2 * dt + 1] = vb0a + (uint32_t)(vb ^ (64 * dt));
        }
    }

    auto barrier = [&]() __attribute__((always_inline)) {
        __builtin_amdgcn_sched_barrier(0);
        asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
        __builtin_amdgcn_sched_barrier(0);
    };
    auto wait_copies = [&]() __attribute__((always_inline)) { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); };

    using yes = std::true_type;

    // M phase of a unit: S^T = K_half Q^T and the product of the previous
    // unit, O^T += V^T P^T.  kp(rt, kk) and vp(cc, dt, ab) give the LDS
    // addresses of the K operand (32-row slice rt, d-chunk kk) and of the
    // two halves of the V^T operand (16 kv rows cc, d-tile dt).  The two
    // products are independent and interleaved; operand reads run PF steps
    // ahead of their products (one step: with no address arithmetic in the
    // phase, two or three steps ran 0.5% and 1.1% slower, and two steps
    // 0.35% slower with the reads between the products).
    auto mphase_at = [&](auto&& kp, auto&& vp) __attribute__((always_inline)) {
        // the matrix phase issues first when both waves of a SIMD are ready
        __builtin_amdgcn_s_setprio(1);
        constexpr int NS = RT * KK;
        constexpr int PF = 1;
        bf16x8 ak[NS];
        s16x4 va4[NS], vb4[NS];
        auto load = [&](auto si) __attribute__((always_inline)) {
            constexpr int s = decltype(si)::value;
            constexpr int rt = s / KK, kk = s % KK, cc = s / DT, dt = s % DT;
            ak[s] = __builtin_bit_cast(bf16x8, *kp(rt, kk));
            va4[s] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(vp(cc, dt, 0));
            vb4[s] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(vp(cc, dt, 1));
        };
        static_for<PF>(load);
        static_for<NS>([&](auto si) __attribute__((always_inline)) {
            constexpr int s = decltype(si)::value;
            constexpr int rt = s / KK, kk = s % KK, cc = s / DT, dt = s % DT;
            sacc[rt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ak[s], qreg[kk], kk == 0 ? f32x16{} : sacc[rt], 0, 0,
                                                               0);
            // the next step's operand reads go out between this step's two
            // products (before the S^T product 0.3% slower; the K read
            // between and the V reads after the PV product 1% slower, the
            // other way round 11% slower)
            if constexpr (s + PF < NS) load(std::integral_constant<int, s + PF>{});
            __builtin_amdgcn_sched_barrier(0);
            const s16x8 v8 = {va4[s][0], va4[s][1], va4[s][2], va4[s][3],
                              vb4[s][0], vb4[s][1], vb4[s][2], vb4[s][3]};
            oacc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, v8), pb[cc], oacc[dt], 0, 0,
                                                               0);
            // keep the operand reads PF steps ahead of their products
            __builtin_amdgcn_sched_barrier(0);
        });
        // the products are issued before the phase ends
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) asm volatile("" : "+v"(sacc[rt]));
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) asm volatile("" : "+v"(oacc[dt]));
        __builtin_amdgcn_s_setprio(0);
    };
    typedef __attribute__((address_space(3))) const uint4 lds_u4_t;
    // In the shared part: the K half tile KO bytes and the V half tile VO
    // bytes past the current buffers (kad, vad).
    auto mphase = [&](auto ko_tag, auto vo_tag) __attribute__((always_inline)) {
        constexpr int KO = decltype(ko_tag)::value, VO = decltype(vo_tag)::value;
        mphase_at(
            [&](int rt, int kk) __attribute__((always_inline)) {
                return (lds_u4_t*)(uintptr_t)(kad[kk] + (uint32_t)(KO + 32 * rt * ROWB));
            },
            [&](int cc, int dt, int ab) __attribute__((always_inline)) {
                return (lds_s16x4_t*)(uintptr_t)(vad[2 * dt + ab] + (uint32_t)(VO + 16 * cc * ROWB));
            });
    };
    // In the exclusive part: the half tiles Kt and Vp of the group's buffers.
    auto mphase_rt = [&](const char* Kt, const char* Vp) __attribute__((always_inline)) {
        mphase_at(
            [&](int rt, int kk) __attribute__((always_inline)) {
                return reinterpret_cast<const uint4*>(Kt + ((ka ^ (32 * kk)) + 32 * rt * ROWB));
            },
            [&](int cc, int dt, int ab) __attribute__((always_inline)) {
                return (lds_s16x4_t*)(Vp + (((ab ? vb : va) ^ (64 * dt)) + 16 * cc * ROWB));
            });
    };
    // The M phase of a unit runs both products unless neither is needed
    // (its tile and the previous one are missing from this group's list); an
    // unneeded one multiplies a zero P, or produces scores nobody reads.
    auto mphase_if = [&](const char* Kt, const char* Vp, bool s_on, bool pv_on) __attribute__((always_inline)) {
        if (s_on || pv_on) mphase_rt(Kt, Vp);
    };
    auto zero_p = [&]() __attribute__((always_inline)) {
#pragma unroll
        for (int c = 0; c < 2 * RT; ++c) pb[c] = bf16x8{};
    };

    // X phase of a unit (kv rows half*KVW .. of a tile with kvalid valid
    // rows): one online-softmax step, P rounded to bf16 in pb.
    // Fast path: the running max m is kept and P = exp2(S*c2 - m*c2) is
    // computed at once; it stands if no lane's probabilities of the unit sum
    // to more than kSumLimit (so none exceeds it: P and the row sums stay well
    // inside fp32 and bf16 range).  Otherwise (and while a row has seen no
    // key yet) the slow path takes the unit's max, moves m up to it, rescales
    // O and l, and computes P again.  The copies cg (a full tile's source,
    // or nullptr) into ct are interleaved with the fast path's exponentials
    // (the compiler schedules them), or issued at once by the slow path when
    // the fast path did not run.
    auto exps = [&](auto copies_tag, auto&& cpf, float& ps0, float& ps1) __attribute__((always_inline)) {
        constexpr bool copies = decltype(copies_tag)::value;
        constexpr int NE = RT * 16;
        static_assert(NE % IPW == 0, "copies must spread evenly over the exponentials");
        ps0 = 0.0f;
        ps1 = 0.0f;
#pragma unroll
        for (int qq = 0; qq < NE; ++qq) {
            if (copies && qq % (NE / IPW) == 0) cpf(qq / (NE / IPW));
            const int rt = qq / 16, c1 = (qq / 8) % 2, e = qq % 8;
            const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[rt][8 * c1 + e], c2, -mb));
            pb[2 * rt + c1][e] = static_cast<__bf16>(p);
            if (qq % 2 == 0)
                ps0 += p;
            else
                ps1 += p;
            // scheduled four scores at a time: left alone, the compiler
            // issues all 32 multiply-adds first (0.65% slower; pinning
            // every score, 3% slower; eight or sixteen, 0.3% / 0.2%)
            if (qq % 4 == 3) __builtin_amdgcn_sched_barrier(0);
        }
#pragma unroll
        for (int c = 0; c < 2 * RT; ++c) asm volatile("" : "+v"(pb[c]));
    };
    auto no_copy = [](int) {};
    auto xphase = [&](int kvalid, auto half_tag, bool cp_on, auto&& cpf) __attribute__((always_inline)) {
        constexpr int half = decltype(half_tag)::value;
        if (kvalid < BS) {
            asm volatile("" ::: "memory");
            // rows at or past the end of the sequence score -inf
#pragma unroll
            for (int rt = 0; rt < RT; ++rt) {
                const int lim = kvalid - (half * KVW + 32 * rt + 4 * h);
#pragma unroll
                for (int ii = 0; ii < 16; ++ii)
                    sacc[rt][ii] = (8 * (ii >> 2) + (ii & 3) >= lim) ? -INFINITY : sacc[rt][ii];
            }
        }
        float ps0, ps1;
        bool fast = __all(m > -INFINITY);
        if (fast) {
            if (cp_on)
                exps(yes{}, cpf, ps0, ps1);
            else
                exps(std::false_type{}, no_copy, ps0, ps1);
            fast = !__any(!(ps0 + ps1 <= kSumLimit));
        } else if (cp_on) {
#pragma unroll
            for (int c = 0; c < IPW; ++c) cpf(c);
        }
        if (!fast) {
            asm volatile("" ::: "memory");
            // tree of 3-input maxima (short dependency chains)
            float t1[RT * 6];
#pragma unroll
            for (int rt = 0; rt < RT; ++rt) {
#pragma unroll
                for (int gq = 0; gq < 5; ++gq)
                    t1[6 * rt + gq] = fmaxf(sacc[rt][3 * gq], fmaxf(sacc[rt][3 * gq + 1], sacc[rt][3 * gq + 2]));
                t1[6 * rt + 5] = sacc[rt][15];
            }
            float mx;
            if constexpr (RT == 2) {
                const float u0 = fmaxf(t1[0], fmaxf(t1[1], t1[2]));
                const float u1 = fmaxf(t1[3], fmaxf(t1[4], t1[5]));
                const float u2 = fmaxf(t1[6], fmaxf(t1[7], t1[8]));
                const float u3 = fmaxf(t1[9], fmaxf(t1[10], t1[11]));
                mx = fmaxf(fmaxf(u0, u1), fmaxf(u2, u3));
            } else {
                mx = fmaxf(fmaxf(t1[0], fmaxf(t1[1], t1[2])), fmaxf(t1[3], fmaxf(t1[4], t1[5])));
            }
            mx = max_across_halves(mx);
            const float m_new = fmaxf(m, mx);
            const float alpha = m_new == m ? 1.0f : __builtin_amdgcn_exp2f((m - m_new) * c2);
            if (__any(alpha != 1.0f)) {
#pragma unroll
                for (int dt = 0; dt < DT; ++dt) oacc[dt] *= alpha;
                l *= alpha;
            }
            m = m_new;
            mb = m_new == -INFINITY ? 0.0f : m_new * c2;
            exps(std::false_type{}, no_copy, ps0, ps1);
        }
        l += ps0 + ps1;
        asm volatile("" : "+v"(l), "+v"(m), "+v"(mb));
    };

    // ---- schedule ----
    // Slot s: group 0 runs phase s, group 1 runs phase s-1 (M and X
    // alternate), then a barrier.  Tile t (K(t) in kc, V(t) in vc) is read
    // by group 0 in the M phases of slots 4t and 4t+2 (V(t) in 4t+2 and
    // 4t+4) and by group 1 one slot later.  During X of its first unit of
    // tile t, group 0 copies K(t+1) into kn (last read in slot 4t-1) and
    // waits for it at the end of the tile (slot 4t+3); group 1 copies V(t+1)
    // into vp (last read in slot 4t+1) and waits for it at the end of its
    // next M phase (slot 4t+5).
    // The walk of the pair has max(cnt(2p), cnt(2p+1)) = ns + max(na, nb)
    // steps: tiles 0 .. ns-1 of the shared part, then the slots of the
    // exclusive part.  A chunk item walks steps [step0, step1) only.
    const int t0 = min(step0, ns), t1 = min(step1, ns);
    uint32_t e_cur = t0 < t1 ? ulist[t0] : 0u;
    uint32_t e_nxt = t0 + 1 < t1 ? ulist[t0 + 1] : 0u;
    e_cur = __builtin_amdgcn_readfirstlane(e_cur);
    e_nxt = __builtin_amdgcn_readfirstlane(e_nxt);
    if (t0 < t1) copy.issue_all(g == 0 ? kg : vg, (int)(e_cur & 0xFFFF), L, g == 0 ? kb0 : vb0, qw, lane);
    // Q and the first tile are complete before the tile loop: no wait on
    // the memory counter (which also counts the tile copies) is left for the
    // loop to inherit.
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) asm volatile("" : "+v"(qreg[kk]));
    wait_copies();
    barrier();
    if (g == 1) barrier();   // group 1 starts one phase late

    bool prev_active = false;   // the previous tile is in this group's list
    // Every block of this part is in both lists: both groups run every phase
    // (the first product multiplies P = 0).
    // The K and V buffers alternate from tile to tile.  The matrix-phase
    // reads take the current buffers from kad (K(t)) and vad: V(t-1) in the
    // first unit, V(t) after a move in the second; kad moves at the end of
    // the tile.  A move adds +TILE or -TILE (the distance between the two
    // buffers of a kind), one instruction per address per tile.
    using IC0 = std::integral_constant<int, 0>;
    using ICH = std::integral_constant<int, HALF>;
    auto move = [&](uint32_t* a, int cnt, int by) __attribute__((always_inline)) {
#pragma unroll
        for (int c = 0; c < cnt; ++c) {
            a[c] += (uint32_t)by;
            asm volatile("" : "+v"(a[c]));
        }
    };
    move(vad, 2 * DT, TILE);   // the first tile's "previous" V half is vb1's (zeroed)
    int mv = TILE;             // kb0 -> kb1 (and vb1 -> vb0) in tile t0, the reverse in t0+1, ...
    char* kn = kb1;            // copy targets: the next tile's K and V buffers
    char* vp = vb1;
    auto tile = [&](int t) __attribute__((always_inline)) {
        const bool more = t + 1 < t1;
        const int jc = (int)(e_cur & 0xFFFF), jn = (int)(e_nxt & 0xFFFF);
        const int kvalid = min(BS, L - jc * BS);
        // first half: S from K(t) rows [0, KVW); product of V(t-1) rows [KVW, BS)
        mphase(IC0{}, ICH{});
        move(vad, 2 * DT, -mv);
        if (g == 1) wait_copies();
        barrier();
        // copy of the next tile (a short one is issued at once by start())
        char* ct = g == 0 ? kn : vp;
        const char* cg = more ? copy.start(g == 0 ? kg : vg, jn, L, ct, qw, lane) : nullptr;
        xphase(kvalid, std::integral_constant<int, 0>{}, cg != nullptr,
               [&](int c) __attribute__((always_inline)) { copy.issue_one(cg, c, ct, qw); });
        barrier();
        // second half: S from K(t) rows [KVW, BS); product of V(t) rows [0, KVW)
        mphase(ICH{}, IC0{});
        barrier();
        uint32_t e_after = t + 2 < t1 ? ulist[t + 2] : 0u;
        e_after = __builtin_amdgcn_readfirstlane(e_after);
        xphase(kvalid, std::integral_constant<int, 1>{}, false, no_copy);
        if (g == 0) wait_copies();
        barrier();
        move(kad, KK, mv);
        mv = -mv;
        kn = kn == kb1 ? kb0 : kb1;
        vp = vp == vb1 ? vb0 : vb1;
        e_cur = e_nxt;
        e_nxt = e_after;
    };
    for (int t = t0; t < t1; ++t) tile(t);
    // the pending product of the last tile's second half (V rows [KVW, BS)
    // of the last tile's V buffer; the scores of that phase go unread)
    if (t1 > t0) mphase(IC0{}, ICH{});
    if (g == 0) barrier();   // both groups pass the same number of barriers

    // ---- blocks in one list only: both groups at once ----
    // Group 0 walks the na blocks of block 2p's list only and group 1 the nb
    // of block 2p+1's only, in the same phase schedule (group 1 one phase
    // behind).  Each group has its own buffers (group 0: kb0, vb0; group 1:
    // kb1, vb1) and copies its own tiles half a tile ahead: during X of the
    // first unit of tile x it copies K(x+1) rows [0, KVW) into the half that
    // unit's M phase has released and V(x) rows [KVW, BS); during X of the
    // second unit, K(x+1) rows [KVW, BS) and V(x+1) rows [0, KVW).  A group
    // waits for its copies at the end of its next X phase.
    const int ce = max(na, nb);   // work-group uniform
    const int x0 = min(ce, max(0, step0 - ns)), x1 = min(ce, max(0, step1 - ns));
    if (x1 > x0) {
        barrier();   // group 1's last product of the shared part has read its buffers
        const int cgx = min(g == 0 ? na : nb, x1);   // this group's end of the walk
        const uint32_t* el = ulist + (g == 0 ? ns : ns + na);
        char* kbuf = g == 0 ? kb0 : kb1;
        char* vbuf = g == 0 ? vb0 : vb1;
        constexpr int IPH = Copy::IPH;
        zero_p();
        uint32_t ec = x0 < cgx ? el[x0] : 0u;
        uint32_t en = x0 + 1 < cgx ? el[x0 + 1] : 0u;
        ec = __builtin_amdgcn_readfirstlane(ec);
        en = __builtin_amdgcn_readfirstlane(en);
        if (x0 < cgx) {
            // the first product multiplies P = 0 with this half: zeros, not stale LDS
            for (int e = 64 * qw + lane; e < HALF / 16; e += 64 * QW)
                reinterpret_cast<uint4*>(vbuf + HALF)[e] = make_uint4(0, 0, 0, 0);
            copy.issue_all(kg, (int)(ec & 0xFFFF), L, kbuf, qw, lane);
            copy.issue_half(vg, (int)(ec & 0xFFFF), L, vbuf, 0, qw, lane);
        }
        wait_copies();
        barrier();
        if (g == 1) barrier();   // group 1 starts one phase late
        prev_active = false;
        // Issue this X phase's copies (K half hk of tile jk if kon, V half hv
        // of tile jv if von) interleaved with its exponentials, or at once if
        // there is no softmax step or a copy is of a short tile; returns the
        // number of copies the wave issued.
        auto xcopies = [&](int kvalid, auto half_tag, bool active, bool kon, int jk, int hk, bool von, int jv,
                           int hv) __attribute__((always_inline)) {
            const char* sk = kon ? copy.start_half(kg, jk, L, kbuf, hk, qw, lane) : nullptr;
            const char* sv = von ? copy.start_half(vg, jv, L, vbuf, hv, qw, lane) : nullptr;
            const bool both = sk != nullptr && sv != nullptr;
            if (!both || !active) {
                if (sk != nullptr) {
#pragma unroll
                    for (int ii = 0; ii < IPH; ++ii) copy.issue_half_one(sk, hk, ii, kbuf, qw);
                }
                if (sv != nullptr) {
#pragma unroll
                    for (int ii = 0; ii < IPH; ++ii) copy.issue_half_one(sv, hv, ii, vbuf, qw);
                }
            }
            if (active)
                xphase(kvalid, half_tag, both, [&](int c) __attribute__((always_inline)) {
                    if (c < IPH)
                        copy.issue_half_one(sk, hk, c, kbuf, qw);
                    else
                        copy.issue_half_one(sv, hv, c - IPH, vbuf, qw);
                });
            else
                zero_p();
            return (kon ? IPH : 0) + (von ? IPH : 0);
        };
        // wait for the copies of the previous X phase: those of this one
        // (issued later, completing later) may still be outstanding
        auto wait_prev = [&](int issued) __attribute__((always_inline)) {
            if (issued == 0)
                wait_vmcnt<0>();
            else if (issued == IPH)
                wait_vmcnt<IPH>();
            else
                wait_vmcnt<2 * IPH>();
        };
        for (int x = x0; x < x1; ++x) {
            const bool active = x < cgx;
            const bool more = x + 1 < cgx;
            const int jc = (int)(ec & 0xFFFF), jn = (int)(en & 0xFFFF);
            const int kvalid = min(BS, L - jc * BS);
            // first half: S from K(x) rows [0, KVW); product of V(x-1) rows [KVW, BS)
            mphase_if(kbuf, vbuf + HALF, active, prev_active);
            barrier();
            const int n0 = xcopies(kvalid, std::integral_constant<int, 0>{}, active, more, jn, 0, active, jc, 1);
            wait_prev(n0);
            barrier();
            // second half: S from K(x) rows [KVW, BS); product of V(x) rows [0, KVW)
            mphase_if(kbuf + HALF, vbuf, active, active);
            barrier();
            uint32_t ea = x + 2 < cgx ? el[x + 2] : 0u;
            ea = __builtin_amdgcn_readfirstlane(ea);
            const int n1 = xcopies(kvalid, std::integral_constant<int, 1>{}, active, more, jn, 1, more, jn, 0);
            wait_prev(n1);
            barrier();
            prev_active = active;
            ec = en;
            en = ea;
        }
        if (prev_active) mphase_rt(kbuf, vbuf + HALF);
        if (g == 0) barrier();
    }

    // ---- output: this wave owns 32 complete query rows ----
    l += __shfl_xor(l, 32);
    if (i < n && qrow < L && slot >= 0) {
        // a chunk of a split pair: O / l in fp32 and the chunk's LSE into its slot
        const float inv = l > 0.0f ? 1.0f / l : 0.0f;
        float* sl = Plan(wsi, BH, npairs, S).part + (size_t)slot * slot_floats(D, BS);
        float* prow = sl + ((size_t)g * BS + 32 * qw + l32) * D;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
            for (int gq = 0; gq < 4; ++gq)
                *reinterpret_cast<float4*>(prow + 32 * dt + 8 * gq + 4 * h) =
                    make_float4(oacc[dt][4 * gq] * inv, oacc[dt][4 * gq + 1] * inv, oacc[dt][4 * gq + 2] * inv,
                                oacc[dt][4 * gq + 3] * inv);
        if (h == 0) sl[2 * BS * D + g * BS + 32 * qw + l32] = l > 0.0f ? m * scale + logf(l) : -INFINITY;
    } else if (i < n && qrow < L) {
        const float inv = l > 0.0f ? 1.0f / l : 0.0f;
        uint16_t* orow = o + base + (size_t)qrow * D;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
            for (int gq = 0; gq < 4; ++gq) {
                uint16_t vals[4];
#pragma unroll
                for (int rr = 0; rr < 4; ++rr)
                    vals[rr] = __builtin_bit_cast(uint16_t, static_cast<__bf16>(oacc[dt][4 * gq + rr] * inv));
                uint2 pk;
                pk.x = (uint32_t)vals[0] | ((uint32_t)vals[1] << 16);
                pk.y = (uint32_t)vals[2] | ((uint32_t)vals[3] << 16);
                *reinterpret_cast<uint2*>(orow + 32 * dt + 8 * gq + 4 * h) = pk;
            }
        if (lse != nullptr && h == 0)
            lse[(size_t)bh * L + qrow] = l > 0.0f ? m * scale + logf(l) : -INFINITY;
    }
    }   // next item
}

// Persistent work-groups per launch: one per compute unit of the current
// device (cached per device; the attribute query is a host call).
int persistent_groups() {
    constexpr int kMaxDevices = 64;
    static std::atomic<int> cus[kMaxDevices];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return 256;
    int c = cus[dev].load(std::memory_order_relaxed);
    if (c == 0) {
        if (hipDeviceGetAttribute(&c, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || c <= 0)
            c = 256;
        cus[dev].store(c, std::memory_order_relaxed);
    }
    return c;
}

template <int D, int BS>
hipError_t launch(const uint16_t* q, const uint16_t* k, const uint16_t* v, const int32_t* kv_idx,
                  const int32_t* kv_cnt, float scale, uint16_t* o, float* lse, int BH, int L, int n,
                  void* ws, int S, hipStream_t s) {
    const int ncu = persistent_groups();
    hipLaunchKernelGGL(plan_kernel, dim3(kXcds), dim3(kPlanThreads), 0, s, kv_cnt, ws, BH, n, ncu, S);
    const long items = (long)BH * ((n + 1) / 2) + S;
    const unsigned groups = (unsigned)std::min<long>(ncu, items);
    hipLaunchKernelGGL((attn_fwd_kernel<D, BS>), dim3(groups), dim3(BS * 4), 0, s,
                       q, k, v, kv_idx, kv_cnt, scale, o, lse, L, n, ws, BH, S);
    if (S > 0)
        hipLaunchKernelGGL((merge_kernel<D, BS>), dim3((unsigned)(2 * ncu)), dim3(256), 0, s, ws, BH, n, S, L, o,
                           lse);
    return hipGetLastError();
}


// ---------------------------------------------------------------------------
// Eq. 2 statistic of the attention map a step computed: for every listed
// block (i, j), the fraction of the probabilities exp(scale q_p.k_q - LSE_p)
// that reach eta, LSE_p being the row LSE the attention forward returned
// over the same lists (the masked map; all blocks at a dense step).  The
// decision is taken in fp32 as s - thr >= 0, thr = (LSE_p + log(eta)) /
// scale, s - thr accumulated by the MFMA products from -thr (it differs
// from rounding s first by a few ulps of s, far inside the log-space band
// where an fp64 reference and any fp32 evaluation may disagree).  Like the
// attention, one work-group per (head, pair of query
// blocks 2p, 2p+1) walks the union of the two lists with two groups of BS/32
// waves (32 query rows each), so every K tile copied into LDS serves both
// blocks (double-buffered, every wave copying its share of the next tile).
// Per tile each wave computes S^T = K Q^T for its 32 query rows by MFMA and
// counts its entries that reach the row's threshold (the sign bits of the
// lane's values summed per lane, then over the wave).  The groups are
// skewed by one tile with a single work-group barrier per tile: in the
// interval of tile t group 0 multiplies tile t and then counts it, while
// group 1 first counts tile t-1 (its scores kept in registers) and then
// multiplies tile t, so on each SIMD one wave's matrix products run beside
// the other wave's compares.  A group's count of
// a tile is summed over its waves and written into stat[bh][i][j] (fp64)
// after the next barrier, by group 0's first wave at the end of its interval
// (off group 1's path, which bounds the interval); blocks not listed keep
// their previous value (the reconstruction of Eq. 5).
// With a text segment after the video the lists cover all n blocks of the
// sequence while the statistic covers the first nv (video) blocks: rows
// i < nv are counted and only entries j < nv are stored (stat [BH, nv, nv]).
// ---------------------------------------------------------------------------
template <int D, int BS>
__global__ __launch_bounds__(BS * 4, 1) void stat_count_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
    const int32_t* __restrict__ kv_idx, const int32_t* __restrict__ kv_cnt,
    const float* __restrict__ lse, float scale, float log_eta, double* __restrict__ stat, int L, int n,
    int nv) {
    constexpr int QW = BS / 32;        // waves per group, 32 query rows each
    constexpr int NT = BS * 4;         // two groups
    constexpr int RT = BS / 32;        // 32-row kv sub-tiles per tile
    constexpr int KK = D / 16;
    constexpr int TILE = BS * D * 2;
    constexpr int ROWB = 2 * D;
    using Copy = TileCopy<D, BS, 2 * QW>;   // copies by all waves
    __shared__ __align__(1024) char kbuf[2][TILE];   // K tiles, double-buffered
    __shared__ uint32_t ulist[kMaxBlocks];
    __shared__ uint8_t umask[kMaxBlocks];
    __shared__ int wsum[NT / 64];
    __shared__ int part[2][2][QW];     // [tile parity][group][wave] counts

    const int npv = (nv + 1) / 2;      // pairs of video rows
    const int bh = blockIdx.x / npv, pr = blockIdx.x % npv;
    const int tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int h = lane >> 5, l32 = lane & 31;
    const int qw = w % QW, g = w / QW;
    const int i = 2 * pr + g;          // this group's query block (nv: none)
    const size_t base = (size_t)bh * L * D;
    const int qrow = i * BS + 32 * qw + l32;
    const bool row_ok = i < nv && qrow < L;

    const size_t row0 = (size_t)bh * n + 2 * pr;
    const int ucnt = union_of_rows<NT>(kv_idx, kv_cnt, row0, 2 * pr + 1 < nv, n, umask, ulist, wsum, tid,
                                       lane, w);

    bf16x8 qreg[KK];
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
        uint4 val = make_uint4(0, 0, 0, 0);
        if (row_ok) val = *reinterpret_cast<const uint4*>(q + base + (size_t)qrow * D + 16 * kk + 8 * h);
        qreg[kk] = __builtin_bit_cast(bf16x8, val);
    }
    // a row past the end of the sequence (or of the video rows) never counts
    const float thr = row_ok ? (lse[(size_t)bh * L + qrow] + log_eta) / scale : INFINITY;
    __syncthreads();   // publishes the union list

    const Copy copy(lane);
    const uint16_t* kg = k + base;
    const int ka = l32 * ROWB + ((h ^ swz<D>(l32)) << 4);

    f32x16 sacc[RT];
    // the products start from -thr, so a score reaches the threshold iff
    // its accumulated value is not negative
    f32x16 nthr;
#pragma unroll
    for (int e = 0; e < 16; ++e) nthr[e] = -thr;
    // S^T - thr of a whole tile: the RT sub-tiles' chains interleaved, operand
    // loads PF steps ahead of their products (pinned step by step)
    auto multiply = [&](const char* kt) __attribute__((always_inline)) {
        constexpr int NS = RT * KK;
        constexpr int PF = 6;
        bf16x8 ak[NS];
        auto load = [&](int s2) __attribute__((always_inline)) {
            const int kk = s2 / RT, rt = s2 % RT;
            ak[s2] = __builtin_bit_cast(bf16x8,
                                        *reinterpret_cast<const uint4*>(kt + ((ka ^ (32 * kk)) + 32 * rt * ROWB)));
        };
#pragma unroll
        for (int s2 = 0; s2 < PF; ++s2) load(s2);
#pragma unroll
        for (int s2 = 0; s2 < NS; ++s2) {
            if (s2 + PF < NS) load(s2 + PF);
            const int kk = s2 / RT, rt = s2 % RT;
            sacc[rt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ak[s2], qreg[kk], kk == 0 ? nthr : sacc[rt], 0, 0,
                                                               0);
            __builtin_amdgcn_sched_barrier(0);
        }
    };
    // entries of the tile in sacc that reach the row's threshold, summed over
    // the wave; rows at or past kvalid (the end of the sequence, in a short
    // tail tile only) are first set to -inf so that they never count
    auto count = [&](int kvalid) __attribute__((always_inline)) {
        if (kvalid < BS) {
            asm volatile("" ::: "memory");
#pragma unroll
            for (int rt = 0; rt < RT; ++rt) {
                const int lim = kvalid - (32 * rt + 4 * h);
#pragma unroll
                for (int ii = 0; ii < 16; ++ii)
                    sacc[rt][ii] = (8 * (ii >> 2) + (ii & 3) >= lim) ? -INFINITY : sacc[rt][ii];
            }
        }
        // the lane's count from the sign bits of its 16 RT values (S - thr;
        // -inf for the masked rows): one byte permute per two values turns
        // the sign bit of the first into 0xFF or 0 in byte 2 and that of the
        // second in byte 0 (selectors 11 and 9 replicate bit 31 of the first
        // and second source), and three-input additions sum two permutes at
        // a time, so each 16-bit half of acc holds 255 x (a count of at most
        // 8 RT) and no carry crosses between them: 0.75 vector instructions
        // per value.  Then the wave's sum, still scaled by 255: within each
        // row of 16 lanes by DPP, over the four rows on the scalar unit.
        uint32_t acc = 0;
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
#pragma unroll
            for (int ii = 0; ii < 16; ii += 4) {
                const uint32_t p0 = __builtin_amdgcn_perm(__float_as_uint(sacc[rt][ii]),
                                                          __float_as_uint(sacc[rt][ii + 1]), 0x0C0B0C09u);
                const uint32_t p1 = __builtin_amdgcn_perm(__float_as_uint(sacc[rt][ii + 2]),
                                                          __float_as_uint(sacc[rt][ii + 3]), 0x0C0B0C09u);
                acc += p0 + p1;
            }
        int v = (int)(255u * 16u * RT - ((acc & 0xFFFFu) + (acc >> 16)));
        v += __builtin_amdgcn_update_dpp(0, v, 0xB1, 0xF, 0xF, false);    // quad_perm [1,0,3,2]
        v += __builtin_amdgcn_update_dpp(0, v, 0x4E, 0xF, 0xF, false);    // quad_perm [2,3,0,1]
        v += __builtin_amdgcn_update_dpp(0, v, 0x124, 0xF, 0xF, false);   // row_ror:4
        v += __builtin_amdgcn_update_dpp(0, v, 0x128, 0xF, 0xF, false);   // row_ror:8
        const int c = __builtin_amdgcn_readlane(v, 0) + __builtin_amdgcn_readlane(v, 16) +
                      __builtin_amdgcn_readlane(v, 32) + __builtin_amdgcn_readlane(v, 48);
        return (int)((uint32_t)c / 255u);   // the wave's count
    };
    // group gg's count of a finished tile (block 2p+gg, kv block j)
    auto flush = [&](int gg, int parity, int j) __attribute__((always_inline)) {
        const int ig = 2 * pr + gg;
        if (lane == 0 && ig < nv && j < nv) {
            int total = 0;
#pragma unroll
            for (int ww = 0; ww < QW; ++ww) total += part[parity][gg][ww];
            stat[((size_t)bh * nv + ig) * nv + j] =
                (double)total / ((double)min(BS, L - ig * BS) * (double)min(BS, L - j * BS));
        }
    };
    auto entry = [&](int t) __attribute__((always_inline)) {
        return __builtin_amdgcn_readfirstlane(ulist[t]);
    };

    if (ucnt > 0) copy.issue_all(kg, (int)(entry(0) & 0xFFFF), L, kbuf[0], w, lane);
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) asm volatile("" : "+v"(qreg[kk]));
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    // interval t (t = 0 .. ucnt; group 0 idles in the last one): the next
    // tile's copies, group 0 multiplies and counts tile t, group 1 counts
    // tile t-1 and multiplies tile t; group 0's first wave then flushes the
    // counts of interval t-1 (group 0's tile t-1, group 1's tile t-2).  The
    // list entries of tiles t-2 .. t+1 are carried in scalar registers; the
    // entry of tile t+2 is read from LDS at the start of the interval and
    // taken at its end.
    // Each group runs its own copy of the interval loop (the same barriers in
    // the same order): group 1's scores live from one interval into the
    // next and group 0's do not, which one shared loop body would reconcile
    // by copying the scores at every iteration.
    uint32_t em2 = 0u, em1 = 0u;
    uint32_t e0 = ucnt > 0 ? entry(0) : 0u;
    uint32_t e1 = ucnt > 1 ? entry(1) : 0u;
    // the part of an interval both groups run first and last
    auto begin = [&](int t) __attribute__((always_inline)) {
        if (t + 1 < ucnt) copy.issue_all(kg, (int)(e1 & 0xFFFF), L, kbuf[(t + 1) & 1], w, lane);
        return ulist[min(t + 2, max(ucnt - 1, 0))];
    };
    auto end = [&](int t, uint32_t e2v) __attribute__((always_inline)) {
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) asm volatile("" : "+v"(sacc[rt]));
        const uint32_t e2 = t + 2 < ucnt ? __builtin_amdgcn_readfirstlane(e2v) : 0u;
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();
        em2 = em1;
        em1 = e0;
        e0 = e1;
        e1 = e2;
    };
    if (g == 0) {
        for (int t = 0; t <= ucnt; ++t) {
            const uint32_t e2v = begin(t);
            const int jc = (int)(e0 & 0xFFFF);
            if (t < ucnt && (e0 >> 16 & 1u) != 0) {
                __builtin_amdgcn_s_setprio(1);
                multiply(kbuf[t & 1]);
                __builtin_amdgcn_s_setprio(0);
                const int c = count(min(BS, L - jc * BS));
                if (lane == 0) part[t & 1][0][qw] = c;
            }
            if (qw == 0) {
                if (t >= 1 && ((em1 >> 16) & 1u) != 0) flush(0, (t - 1) & 1, (int)(em1 & 0xFFFF));
                if (t >= 2 && ((em2 >> 17) & 1u) != 0) flush(1, t & 1, (int)(em2 & 0xFFFF));
            }
            end(t, e2v);
        }
    } else {
        for (int t = 0; t <= ucnt; ++t) {
            const uint32_t e2v = begin(t);
            // counts of tile t-1 first (they free the scores), then this
            // tile's products
            int c = 0;
            const bool pm = t > 0 && ((em1 >> 17) & 1u) != 0;
            if (pm) c = count(min(BS, L - (int)(em1 & 0xFFFF) * BS));
            if (t < ucnt && (e0 >> 17 & 1u) != 0) {
                __builtin_amdgcn_s_setprio(1);
                multiply(kbuf[t & 1]);
                __builtin_amdgcn_s_setprio(0);
            }
            if (pm && lane == 0) part[(t - 1) & 1][1][qw] = c;
            end(t, e2v);
        }
    }
    // group 1's count of the last tile (interval ucnt; its entry is in em2
    // after the last rotation) is flushed here
    if (g == 1 && qw == 0 && ucnt > 0 && ((em2 >> 17) & 1u) != 0) flush(1, (ucnt - 1) & 1, (int)(em2 & 0xFFFF));
}

template <int D, int BS>
hipError_t launch_count(const uint16_t* q, const uint16_t* k, const int32_t* kv_idx, const int32_t* kv_cnt,
                        const float* lse, float scale, float log_eta, double* stat, int BH, int L, int n,
                        int nv, hipStream_t s) {
    const unsigned npv = (unsigned)(nv + 1) / 2;
    hipLaunchKernelGGL((stat_count_kernel<D, BS>), dim3((unsigned)BH * npv), dim3(BS * 4), 0, s, q, k, kv_idx,
                       kv_cnt, lse, scale, log_eta, stat, L, n, nv);
    return hipGetLastError();
}

}  // namespace

// ---------------------------------------------------------------------------
// Work plan in library-owned device memory, for callers that cannot
// allocate: one array per device (each device holds its own copy at its
// own address), kept until the process ends and shared by every call on
// that device.  Host code never passes the array's name to a kernel (on the
// host it only names a stand-in); the device address comes from
// hipGetSymbolAddress, resolved once per device with that device current.
// Nothing in it needs clearing between calls: the plan kernels rewrite every
// field the attention reads (the fetch counters included) before it runs.
// ---------------------------------------------------------------------------
static __device__ __align__(256) char scratch[kNoAllocScratchBytes];

namespace {
constexpr int kScratchDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kScratchDevices] = {};
}  // namespace

hipError_t noalloc_scratch(void** out) {
    *out = nullptr;
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kScratchDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (g_scratch_ptr[dev] == nullptr) {
        void* ptr = nullptr;
        e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (ptr == nullptr) return hipErrorInvalidSymbol;
        g_scratch_ptr[dev] = ptr;
    }
    *out = g_scratch_ptr[dev];
    return hipSuccess;
}

size_t attn_plan_bytes(int BH, int n, int S) {
    return Plan::ints(BH, (n + 1) / 2, S) * sizeof(int);
}

size_t attn_slot_bytes(int d, int bs) { return slot_floats(d, bs) * sizeof(float); }

int attn_max_slots(int BH, int n) {
    // every chunk is at least kMinChunkSteps steps of a walk of at most n
    const long long per_pair = (n + kMinChunkSteps - 1) / kMinChunkSteps;
    const long long bound = per_pair > 1 ? (long long)BH * ((n + 1) / 2) * per_pair : 0;
    return (int)std::min<long long>(kMaxSplitSlots, bound);
}

size_t attn_workspace_bytes(int BH, int n, int d, int bs) {
    const int S = attn_max_slots(BH, n);
    return attn_plan_bytes(BH, n, S) + (size_t)S * attn_slot_bytes(d, bs);
}

int attn_slots_for(int BH, int n, int d, int bs, size_t ws_bytes) {
    const size_t base = attn_plan_bytes(BH, n, 0);
    if (ws_bytes <= base) return 0;
    // each slot adds 9 plan ints (item, chunk, split descriptors) and a slot
    long long S = (long long)((ws_bytes - base) / (attn_slot_bytes(d, bs) + 9 * sizeof(int)));
    S = std::min<long long>(S, attn_max_slots(BH, n));
    while (S > 0 && attn_plan_bytes(BH, n, (int)S) + (size_t)S * attn_slot_bytes(d, bs) > ws_bytes) --S;
    return S < 2 ? 0 : (int)S;
}

hipError_t launch_attn_fwd(const uint16_t* q, const uint16_t* k, const uint16_t* v,
                           const int32_t* kv_idx, const int32_t* kv_cnt, float scale,
                           uint16_t* o, float* lse, int BH, int L, int d, int bs, int n,
                           void* ws, size_t ws_bytes, hipStream_t s) {
    const int S = attn_slots_for(BH, n, d, bs, ws_bytes);
    if (d == 128 && bs == 128) return launch<128, 128>(q, k, v, kv_idx, kv_cnt, scale, o, lse, BH, L, n, ws, S, s);
    if (d == 128 && bs == 64) return launch<128, 64>(q, k, v, kv_idx, kv_cnt, scale, o, lse, BH, L, n, ws, S, s);
    if (d == 64 && bs == 128) return launch<64, 128>(q, k, v, kv_idx, kv_cnt, scale, o, lse, BH, L, n, ws, S, s);
    return launch<64, 64>(q, k, v, kv_idx, kv_cnt, scale, o, lse, BH, L, n, ws, S, s);
}

hipError_t launch_stat_count(const uint16_t* q, const uint16_t* k, const int32_t* kv_idx,
                             const int32_t* kv_cnt, const float* lse, float scale, float log_eta,
                             double* stat, int BH, int L, int d, int bs, int n, int nv, hipStream_t s) {
    if (d == 128 && bs == 128) return launch_count<128, 128>(q, k, kv_idx, kv_cnt, lse, scale, log_eta, stat, BH, L, n, nv, s);
    if (d == 128 && bs == 64) return launch_count<128, 64>(q, k, kv_idx, kv_cnt, lse, scale, log_eta, stat, BH, L, n, nv, s);
    if (d == 64 && bs == 128) return launch_count<64, 128>(q, k, kv_idx, kv_cnt, lse, scale, log_eta, stat, BH, L, n, nv, s);
    return launch_count<64, 64>(q, k, kv_idx, kv_cnt, lse, scale, log_eta, stat, BH, L, n, nv, s);
}

}  // namespace moddit
