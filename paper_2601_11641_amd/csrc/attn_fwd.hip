// Block-sparse attention forward for gfx950 (Eq. 1 with a block mask).
//
// One workgroup per (head, query block i); BS/32 waves, each owning 32 query
// rows.  For every kept key block j of the row's list the K tile and the
// transposed V tile are staged in LDS, and each wave computes
//
//   S^T (BS x 32)  = K_j (BS x D) . Q^T (D x 32)      v_mfma_f32_32x32x16_bf16
//   online softmax over the kv dimension in fp32 registers
//   O^T (D x 32)  += V_j^T (D x BS) . P^T (BS x 32)   v_mfma_f32_32x32x16_bf16
//
// Computing the transposed products puts one query row in the column of
// every lane, so the row max and the rescale of the accumulator are
// per-lane scalars (one cross-half exchange per tile), and the fp32
// probabilities of S^T feed the next MFMA as its B operand without moving
// between lanes: the K rows are loaded in a permuted order that makes the
// accumulator rows of a lane exactly the 8 consecutive kv positions the
// B operand of the PV product expects.
#include "moddit_internal.h"

namespace moddit {
namespace {

typedef __bf16 bf16x8 __attribute__((__vector_size__(8 * sizeof(__bf16))));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr float kLog2e = 1.4426950408889634f;

__device__ inline bf16x8 load_bf16x8(const uint16_t* p) {
    return __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(p));
}

template <int D, int BS>
__global__ __launch_bounds__(BS * 2) void attn_fwd_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
    const uint16_t* __restrict__ v, const int32_t* __restrict__ kv_idx,
    const int32_t* __restrict__ kv_cnt, float scale, uint16_t* __restrict__ o,
    float* __restrict__ lse, int L, int n) {
    constexpr int NT = BS * 2;       // threads
    constexpr int KP = D + 8;        // K tile row pitch (elements)
    constexpr int VP = BS + 8;       // V^T tile row pitch (elements)
    __shared__ __align__(16) uint16_t Ks[BS * KP];
    __shared__ __align__(16) uint16_t Vt[D * VP];

    const int item = blockIdx.x;
    const int bh = item / n, i = item % n;
    const int tid = threadIdx.x, w = tid / 64, lane = tid % 64;
    const int h = lane / 32, l32 = lane % 32;
    const size_t base = (size_t)bh * L * D;
    const int qrow = i * BS + 32 * w + l32;
    const float c2 = scale * kLog2e;

    // Q^T as the B operand: lane holds Q[qrow][16kk + 8h .. +7]
    bf16x8 qreg[D / 16];
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk) {
        if (qrow < L)
            qreg[kk] = load_bf16x8(q + base + (size_t)qrow * D + 16 * kk + 8 * h);
        else
            qreg[kk] = __builtin_bit_cast(bf16x8, make_uint4(0, 0, 0, 0));
    }

    f32x16 oacc[D / 32];
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt) oacc[dt] = f32x16{};
    float m = -INFINITY, lsum = 0.0f;

    // Accumulator row rho of a 32-row tile is kv 32*rt + perm(rho): lane
    // (half h) register ii then holds kv 32*rt + 16*(ii/8) + 8h + (ii%8).
    const int g4 = l32 / 8, hb = (l32 / 4) % 2, r4 = l32 % 4;
    const int krow = 16 * (g4 / 2) + 8 * hb + 4 * (g4 % 2) + r4;

    const int cnt = kv_cnt[item];
    const int32_t* list = kv_idx + (size_t)item * n;
    for (int t = 0; t < cnt; ++t) {
        const int j = list[t];
        const int k0 = j * BS;
        const int kvalid = min(BS, L - k0);
        __syncthreads();
        for (int e = tid; e < BS * (D / 8); e += NT) {
            const int r = e % BS, c = e / BS;
            uint4 kv4 = make_uint4(0, 0, 0, 0), vv4 = make_uint4(0, 0, 0, 0);
            if (r < kvalid) {
                kv4 = *reinterpret_cast<const uint4*>(k + base + (size_t)(k0 + r) * D + c * 8);
                vv4 = *reinterpret_cast<const uint4*>(v + base + (size_t)(k0 + r) * D + c * 8);
            }
            *reinterpret_cast<uint4*>(Ks + r * KP + c * 8) = kv4;
            const uint32_t vw[4] = {vv4.x, vv4.y, vv4.z, vv4.w};
#pragma unroll
            for (int e2 = 0; e2 < 4; ++e2) {
                Vt[(c * 8 + 2 * e2) * VP + r] = static_cast<uint16_t>(vw[e2] & 0xFFFFu);
                Vt[(c * 8 + 2 * e2 + 1) * VP + r] = static_cast<uint16_t>(vw[e2] >> 16);
            }
        }
        __syncthreads();

        f32x16 sacc[BS / 32];
#pragma unroll
        for (int rt = 0; rt < BS / 32; ++rt) {
            sacc[rt] = f32x16{};
#pragma unroll
            for (int kk = 0; kk < D / 16; ++kk) {
                const bf16x8 a = load_bf16x8(Ks + (32 * rt + krow) * KP + 16 * kk + 8 * h);
                sacc[rt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qreg[kk], sacc[rt], 0, 0, 0);
            }
        }
        if (kvalid < BS) {
#pragma unroll
            for (int rt = 0; rt < BS / 32; ++rt)
#pragma unroll
                for (int ii = 0; ii < 16; ++ii) {
                    const int kv = 32 * rt + 16 * (ii / 8) + 8 * h + (ii % 8);
                    if (kv >= kvalid) sacc[rt][ii] = -INFINITY;
                }
        }
        float mx = -INFINITY;
#pragma unroll
        for (int rt = 0; rt < BS / 32; ++rt)
#pragma unroll
            for (int ii = 0; ii < 16; ++ii) mx = fmaxf(mx, sacc[rt][ii]);
        mx = fmaxf(mx, __shfl_xor(mx, 32));
        const float m_new = fmaxf(m, mx);
        const float alpha = exp2f((m - m_new) * c2);
        const float mb = m_new * c2;
        float psum = 0.0f;
#pragma unroll
        for (int rt = 0; rt < BS / 32; ++rt)
#pragma unroll
            for (int ii = 0; ii < 16; ++ii) {
                const float p = exp2f(sacc[rt][ii] * c2 - mb);
                sacc[rt][ii] = p;
                psum += p;
            }
        lsum = lsum * alpha + psum;
        m = m_new;
#pragma unroll
        for (int dt = 0; dt < D / 32; ++dt) oacc[dt] *= alpha;

#pragma unroll
        for (int cc = 0; cc < BS / 16; ++cc) {
            bf16x8 b;
#pragma unroll
            for (int e2 = 0; e2 < 8; ++e2) b[e2] = static_cast<__bf16>(sacc[cc / 2][8 * (cc % 2) + e2]);
#pragma unroll
            for (int dt = 0; dt < D / 32; ++dt) {
                const bf16x8 a = load_bf16x8(Vt + (32 * dt + l32) * VP + 16 * cc + 8 * h);
                oacc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, oacc[dt], 0, 0, 0);
            }
        }
    }

    const float ltot = lsum + __shfl_xor(lsum, 32);
    if (qrow < L) {
        const float inv = ltot > 0.0f ? 1.0f / ltot : 0.0f;
        uint16_t* orow = o + base + (size_t)qrow * D;
#pragma unroll
        for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
            for (int gq = 0; gq < 4; ++gq) {
                const int d0 = 32 * dt + 8 * gq + 4 * h;
                uint16_t vals[4];
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    vals[r] = __builtin_bit_cast(uint16_t,
                                                 static_cast<__bf16>(oacc[dt][4 * gq + r] * inv));
                uint2 pk;
                pk.x = (uint32_t)vals[0] | ((uint32_t)vals[1] << 16);
                pk.y = (uint32_t)vals[2] | ((uint32_t)vals[3] << 16);
                *reinterpret_cast<uint2*>(orow + d0) = pk;
            }
        if (lse != nullptr && h == 0)
            lse[(size_t)bh * L + qrow] = cnt > 0 ? m * scale + logf(ltot) : -INFINITY;
    }
}

}  // namespace

hipError_t launch_attn_fwd(const uint16_t* q, const uint16_t* k, const uint16_t* v,
                           const int32_t* kv_idx, const int32_t* kv_cnt, float scale,
                           uint16_t* o, float* lse, int BH, int L, int d, int bs, int n,
                           hipStream_t s) {
    const dim3 grid((unsigned)BH * n);
    if (d == 128 && bs == 128)
        hipLaunchKernelGGL((attn_fwd_kernel<128, 128>), grid, dim3(256), 0, s, q, k, v, kv_idx,
                           kv_cnt, scale, o, lse, L, n);
    else if (d == 128 && bs == 64)
        hipLaunchKernelGGL((attn_fwd_kernel<128, 64>), grid, dim3(128), 0, s, q, k, v, kv_idx,
                           kv_cnt, scale, o, lse, L, n);
    else if (d == 64 && bs == 128)
        hipLaunchKernelGGL((attn_fwd_kernel<64, 128>), grid, dim3(256), 0, s, q, k, v, kv_idx,
                           kv_cnt, scale, o, lse, L, n);
    else
        hipLaunchKernelGGL((attn_fwd_kernel<64, 64>), grid, dim3(128), 0, s, q, k, v, kv_idx,
                           kv_cnt, scale, o, lse, L, n);
    return hipGetLastError();
}

}  // namespace moddit
