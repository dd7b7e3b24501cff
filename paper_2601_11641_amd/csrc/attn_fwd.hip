// Block-sparse attention forward for gfx950 (Eq. 1 with a block mask).
//
// One workgroup per (head, query block i of BS rows) with 2 * BS/32 waves:
// wave w owns 32 query rows (slice w % (BS/32)) and one half of every
// key/value tile (kv half w / (BS/32)).  Each wave runs its own online
// softmax over its kv halves; the two partial results of a slice are merged
// through LDS at the end.  With 32-row waves everything a wave needs fits in
// 256 registers, so two waves share each SIMD and the hardware interleaves
// one wave's softmax with the other's matrix products.
//
// Per kept key block j of the row's list:
//   * the K and V tiles (BS x D bf16, row-major, 16-byte chunks XOR-swizzled
//     per row) are brought into LDS with global_load_lds_dwordx4 one tile
//     ahead (double buffer), so the copy of tile t+1 overlaps compute on t;
//   * S^T (kv x q) = K . Q^T with v_mfma_f32_32x32x16_bf16: a lane owns one
//     query column, so the row max and the rescale are per-lane scalars;
//   * P = exp2(S * scale*log2e - m) in fp32, rounded to bf16 as the B operand
//     of the next product without moving between lanes;
//   * O^T (d x q) += V^T . P^T, the V^T operand read from the row-major V
//     tile with ds_read_b64_tr_b16 (transposing LDS reads).
// The running max is only moved when a tile's max exceeds it by more than
// 2^8 in probability units, so most tiles skip the accumulator rescale.
#include "moddit_internal.h"

namespace moddit {
namespace {

typedef __bf16 bf16x8 __attribute__((__vector_size__(8 * sizeof(__bf16))));
typedef short s16x4 __attribute__((__vector_size__(4 * sizeof(short))));
typedef short s16x8 __attribute__((__vector_size__(8 * sizeof(short))));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(3))) s16x4 lds_s16x4_t;
typedef __attribute__((address_space(1))) void gbl_void_t;

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kRescaleLog2 = 8.0f;   // lazy-rescale threshold (log2 units)
constexpr int kXcds = 8;               // accelerator complex dies of an MI355X

// XOR pattern applied to the 16-byte chunk index of a tile row.  The MFMA
// operand loads read one chunk column of 8 (or 16) consecutive rows at a
// time, so the pattern must differ in its low 3 (4) bits over any 8 (16)
// aligned consecutive rows; the transposing loads read two adjacent chunks
// (an even/odd pair) of 4 aligned consecutive rows, so bits 1..2 must differ
// over any 4 such rows.  swz(r) = (r&3)<<1 | (r>>2)&1 | (r&8) meets both.
// max(x, x of lane l ^ 32): with x in both operands, v_permlane32_swap
// returns x[l mod 32] and x[l mod 32 + 32] to lane l, i.e. its own value and
// its partner's.
__device__ __forceinline__ float max_across_halves(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                    false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

template <int D>
__device__ __forceinline__ int swz(int row) {
    const int f = ((row & 3) << 1) | ((row >> 2) & 1);
    if constexpr (D == 128)
        return f | (row & 8);
    else
        return f;
}

// Issue this wave's share of the 1-KB direct-to-LDS copies of one BS x D
// tile.  Copy `ins` fills LDS bytes [ins*1024, +1024): lane l writes the
// 16-byte chunk at ins*1024 + 16*l, i.e. row ins*RPI + l/LPR, physical
// chunk l % LPR, which holds logical chunk (l % LPR) ^ swz(row).  The
// per-lane part of the source offset only depends on ins mod 4 (D = 128) or
// not at all (D = 64); it is precomputed in voff.  Rows past the end of the
// sequence (short tail tile) re-read the last valid row: their scores are
// masked and their probabilities are zero.
template <int D, int BS, int NW>
struct TileCopy {
    static constexpr int ROWB = 2 * D;            // bytes per row
    static constexpr int LPR = ROWB / 16;         // lanes per row
    static constexpr int RPI = 64 / LPR;          // rows per 1-KB copy
    static constexpr int IPW = BS * ROWB / 1024 / NW;
    static constexpr int NV = D == 128 ? 4 : 1;
    uint32_t voff[NV];                             // byte offsets, lane part

    __device__ __forceinline__ explicit TileCopy(int lane) {
#pragma unroll
        for (int a = 0; a < NV; ++a) {
            const int row = a * RPI + lane / LPR;  // row mod 16 (D=128) / mod 8 (D=64)
            voff[a] = (uint32_t)((lane / LPR) * ROWB + (((lane % LPR) ^ swz<D>(row)) << 4));
        }
    }

    // g: first element of the head; k0: first row of the tile; w: wave index
    // (wave-uniform); tile: LDS destination (wave-uniform).
    __device__ __forceinline__ void issue(const uint16_t* __restrict__ g, int k0, int kvalid,
                                          char* tile, int w, int lane) const {
        if (kvalid == BS) {
            const char* gt = reinterpret_cast<const char*>(g + (size_t)k0 * D);
#pragma unroll
            for (int ii = 0; ii < IPW; ++ii) {
                const int ins = w * IPW + ii;
                const char* src = gt + (size_t)ins * 1024 + voff[ii % NV];
                __builtin_amdgcn_global_load_lds((gbl_void_t*)src, (lds_void_t*)(tile + ins * 1024),
                                                 16, 0, 0);
            }
        } else {
#pragma unroll
            for (int ii = 0; ii < IPW; ++ii) {
                const int ins = w * IPW + ii;
                const int row = ins * RPI + lane / LPR;
                const int chunk = (lane % LPR) ^ swz<D>(row);
                const uint16_t* src = g + (size_t)(k0 + min(row, kvalid - 1)) * D + chunk * 8;
                __builtin_amdgcn_global_load_lds((gbl_void_t*)src, (lds_void_t*)(tile + ins * 1024),
                                                 16, 0, 0);
            }
        }
    }
};

template <int D, int BS>
__global__ __launch_bounds__(BS * 4, 1) void attn_fwd_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
    const uint16_t* __restrict__ v, const int32_t* __restrict__ kv_idx,
    const int32_t* __restrict__ kv_cnt, float scale, uint16_t* __restrict__ o,
    float* __restrict__ lse, int L, int n) {
    constexpr int QW = BS / 32;        // 32-row query slices
    constexpr int NW = 2 * QW;         // waves: every slice x two kv halves
    constexpr int KVW = BS / 2;        // kv rows per wave per tile
    constexpr int RT = KVW / 32;       // 32-row kv sub-tiles per wave
    constexpr int DT = D / 32;         // 32-row d tiles of O^T
    constexpr int KK = D / 16;         // 16-deep d chunks of S^T
    constexpr int TILE = BS * D * 2;   // bytes per K or V tile
    constexpr int ROWB = 2 * D;
    // Two tile buffers ([K, V] each) as distinct LDS objects: the loop below
    // is unrolled by two so that every copy and every read names its buffer
    // at compile time, which lets the compiler see that the copy into one
    // buffer never aliases the reads of the other (otherwise it waits for the
    // prefetch before the first read of every tile).
    __shared__ __align__(1024) char buf0[2 * TILE];
    __shared__ __align__(1024) char buf1[2 * TILE];

    // Work-group -> (head, query block): dispatch puts work-group b on XCD
    // b % 8.  All XCDs work on the same head at a time (its K/V stays in the
    // shared last-level cache) and each XCD takes a contiguous run of query
    // blocks (neighbouring rows share K/V blocks, so the XCD's L2 serves
    // them).  Padding slots past the last block exit at once.
    const int chunk = (n + kXcds - 1) / kXcds;
    const int xcd = blockIdx.x % kXcds, r = blockIdx.x / kXcds;
    const int bh = r / chunk, i = xcd * chunk + r % chunk;
    if (i >= n) return;
    const int item = bh * n + i;
    const int tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform
    const int h = lane >> 5, l32 = lane & 31;
    const int qw = w % QW, kh = w / QW;
    const size_t base = (size_t)bh * L * D;
    const float c2 = scale * kLog2e;
    const int qrow = i * BS + 32 * qw + l32;

    // Q^T as the B operand of S^T: lane holds Q[qrow][16kk + 8h .. +7]
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
    float m = -INFINITY, l = 0.0f;

    const int cnt = kv_cnt[item];
    const int32_t* list = kv_idx + (size_t)item * n;
    const TileCopy<D, BS, NW> copy(lane);
    if (cnt > 0) {
        const int j0 = list[0];
        const int kv0 = min(BS, L - j0 * BS);
        copy.issue(k + base, j0 * BS, kv0, buf0, w, lane);
        copy.issue(v + base, j0 * BS, kv0, buf0 + TILE, w, lane);
    }

    // Per-lane LDS byte addresses.  The swizzle of every row a lane reads
    // depends only on the lane, so an address is a lane constant XOR a
    // compile-time chunk field, plus a compile-time row offset.
    //   K operand (S^T A operand): row kh*KVW + 32 rt + l32, chunk 2 kk + h
    const int ka = (kh * KVW + l32) * ROWB + ((h ^ swz<D>(l32)) << 4);
    //   V^T operand (transposing reads): rows kv0 + (lane%16)/4 with
    //   kv0 = kh*KVW + 16 cc + 4h (+8), d = 32 dt + 16 ((lane/16)&1) + 4 (lane%4)
    const int s16 = lane & 15, grp = lane >> 4;
    const int tr_row = 4 * h + (s16 >> 2);
    const int c0 = 2 * (grp & 1) + ((s16 & 3) >> 1);
    const int half8 = (s16 & 1) << 3;
    const int va = (kh * KVW + tr_row) * ROWB + ((c0 ^ swz<D>(tr_row)) << 4) + half8;
    const int vb = (kh * KVW + tr_row + 8) * ROWB + ((c0 ^ swz<D>(tr_row + 8)) << 4) + half8;

    // One kv tile: for each 32-row sub-tile of this wave's half, one online
    // softmax step (S^T = K Q^T, softmax, O^T += V^T P^T).  With two waves
    // per SIMD in flight, the hardware overlaps one wave's softmax with the
    // other's products.  The rarely taken branches (short tail tile, rescale)
    // hold an empty volatile asm so the compiler keeps them as branches
    // instead of turning them into unconditional selects and multiplies.
    auto tile_step = [&](const char* Kt, const char* Vt, int kvalid) {
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
            f32x16 s = f32x16{};
#pragma unroll
            for (int kk = 0; kk < KK; ++kk) {
                const bf16x8 a = __builtin_bit_cast(
                    bf16x8, *reinterpret_cast<const uint4*>(Kt + ((ka ^ (32 * kk)) + 32 * rt * ROWB)));
                s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qreg[kk], s, 0, 0, 0);
            }
            if (kvalid < BS) {
                asm volatile("" ::: "memory");
                // rows at or past the end of the sequence score -inf
                const int lim = kvalid - (kh * KVW + 32 * rt + 4 * h);
#pragma unroll
                for (int ii = 0; ii < 16; ++ii)
                    s[ii] = (8 * (ii >> 2) + (ii & 3) >= lim) ? -INFINITY : s[ii];
            }
            float mx = -INFINITY;
#pragma unroll
            for (int ii = 0; ii < 16; ++ii) mx = fmaxf(mx, s[ii]);
            mx = max_across_halves(mx);
            const bool need = (mx - m) * c2 > kRescaleLog2;
            const float m_new = need ? mx : m;
            const float alpha = need ? __builtin_amdgcn_exp2f((m - mx) * c2) : 1.0f;
            const float mb = m_new == -INFINITY ? 0.0f : m_new * c2;
            float ps = 0.0f;
#pragma unroll
            for (int ii = 0; ii < 16; ++ii) {
                const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(s[ii], c2, -mb));
                s[ii] = p;
                ps += p;
            }
            l = l * alpha + ps;
            m = m_new;
            if (__any(need)) {
                asm volatile("" ::: "memory");
#pragma unroll
                for (int dt = 0; dt < DT; ++dt) oacc[dt] *= alpha;
            }
#pragma unroll
            for (int c1 = 0; c1 < 2; ++c1) {
                const int cc = 2 * rt + c1;
                bf16x8 b;
#pragma unroll
                for (int e = 0; e < 8; ++e) b[e] = static_cast<__bf16>(s[8 * c1 + e]);
#pragma unroll
                for (int dt = 0; dt < DT; ++dt) {
                    const s16x4 ta = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                        (lds_s16x4_t*)(Vt + ((va ^ (64 * dt)) + 16 * cc * ROWB)));
                    const s16x4 tb = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                        (lds_s16x4_t*)(Vt + ((vb ^ (64 * dt)) + 16 * cc * ROWB)));
                    const s16x8 v8 = {ta[0], ta[1], ta[2], ta[3], tb[0], tb[1], tb[2], tb[3]};
                    oacc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                        __builtin_bit_cast(bf16x8, v8), b, oacc[dt], 0, 0, 0);
                }
            }
        }
    };

    // tile t lives in `cur`; the copy of tile t+1 goes to `nxt`
    auto step = [&](int t, const char* cur, char* nxt) {
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();
        if (t + 1 < cnt) {
            const int jn = list[t + 1];
            const int kvn = min(BS, L - jn * BS);
            copy.issue(k + base, jn * BS, kvn, nxt, w, lane);
            copy.issue(v + base, jn * BS, kvn, nxt + TILE, w, lane);
        }
        const int j = list[t];
        tile_step(cur, cur + TILE, min(BS, L - j * BS));
    };
    for (int t = 0; t < cnt; t += 2) {
        step(t, buf0, buf1);
        if (t + 1 < cnt) step(t + 1, buf1, buf0);
    }

    // merge the two kv halves of every query slice through LDS
    l += __shfl_xor(l, 32);
    __syncthreads();
    float* mo = reinterpret_cast<float*>(buf0) + qw * (DT * 16 * 64 + 2 * 64);
    if (kh == 1) {
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
            for (int ii = 0; ii < 16; ++ii) mo[(dt * 16 + ii) * 64 + lane] = oacc[dt][ii];
        mo[DT * 16 * 64 + lane] = m;
        mo[DT * 16 * 64 + 64 + lane] = l;
    }
    __syncthreads();
    if (kh == 0) {
        const float mb = mo[DT * 16 * 64 + lane];
        const float lb = mo[DT * 16 * 64 + 64 + lane];
        const float mm = fmaxf(m, mb);
        const float fa = m == -INFINITY ? 0.0f : __builtin_amdgcn_exp2f((m - mm) * c2);
        const float fb = mb == -INFINITY ? 0.0f : __builtin_amdgcn_exp2f((mb - mm) * c2);
        const float ltot = l * fa + lb * fb;
        const float inv = ltot > 0.0f ? 1.0f / ltot : 0.0f;
        if (qrow < L) {
            uint16_t* orow = o + base + (size_t)qrow * D;
#pragma unroll
            for (int dt = 0; dt < DT; ++dt)
#pragma unroll
                for (int gq = 0; gq < 4; ++gq) {
                    uint16_t vals[4];
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const int ii = 4 * gq + r;
                        const float ob = mo[(dt * 16 + ii) * 64 + lane];
                        const float val = (oacc[dt][ii] * fa + ob * fb) * inv;
                        vals[r] = __builtin_bit_cast(uint16_t, static_cast<__bf16>(val));
                    }
                    uint2 pk;
                    pk.x = (uint32_t)vals[0] | ((uint32_t)vals[1] << 16);
                    pk.y = (uint32_t)vals[2] | ((uint32_t)vals[3] << 16);
                    *reinterpret_cast<uint2*>(orow + 32 * dt + 8 * gq + 4 * h) = pk;
                }
            if (lse != nullptr && h == 0)
                lse[(size_t)bh * L + qrow] = ltot > 0.0f ? mm * scale + logf(ltot) : -INFINITY;
        }
    }
}

template <int D, int BS>
hipError_t launch(const uint16_t* q, const uint16_t* k, const uint16_t* v, const int32_t* kv_idx,
                  const int32_t* kv_cnt, float scale, uint16_t* o, float* lse, int BH, int L, int n,
                  hipStream_t s) {
    const unsigned chunk = (unsigned)(n + kXcds - 1) / kXcds;
    hipLaunchKernelGGL((attn_fwd_kernel<D, BS>), dim3((unsigned)BH * chunk * kXcds), dim3(BS * 4), 0, s,
                       q, k, v,
                       kv_idx, kv_cnt, scale, o, lse, L, n);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_attn_fwd(const uint16_t* q, const uint16_t* k, const uint16_t* v,
                           const int32_t* kv_idx, const int32_t* kv_cnt, float scale,
                           uint16_t* o, float* lse, int BH, int L, int d, int bs, int n,
                           hipStream_t s) {
    if (d == 128 && bs == 128) return launch<128, 128>(q, k, v, kv_idx, kv_cnt, scale, o, lse, BH, L, n, s);
    if (d == 128 && bs == 64) return launch<128, 64>(q, k, v, kv_idx, kv_cnt, scale, o, lse, BH, L, n, s);
    if (d == 64 && bs == 128) return launch<64, 128>(q, k, v, kv_idx, kv_cnt, scale, o, lse, BH, L, n, s);
    return launch<64, 64>(q, k, v, kv_idx, kv_cnt, scale, o, lse, BH, L, n, s);
}

}  // namespace moddit
