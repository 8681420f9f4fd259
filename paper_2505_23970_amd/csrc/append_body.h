// KV append for gfx950 (device code shared by the append kernel and the fused
// append-and-plan launch): copy the new tokens' K/V into their pool slots
// (GreenCache §2.2, Fig. 1a step 1: the processed request's KV is saved so a
// later request with the same context can reuse it).
//
// A workgroup takes 16 consecutive packed new tokens of one KV head (the grid
// covers tokens x heads, so a batch of a few thousand tokens still fills the
// GPU). Keys are copied row by row (each 16-byte chunk read once, written once,
// coalesced on both sides). Values go to transposed pages ([D][16]): the 16
// tokens' rows are staged in LDS and written out column-wise, so the 16 lanes
// that write one page row touch 32 consecutive bytes when the tokens share a
// page. Slots whose block id is missing or outside the pool are skipped.
// 8-bit pools store E4M3 codes: each element x becomes the code nearest to
// fl32(x * inv) clamped to [-448, 448] (ties to even; the conversion
// instruction rounds to nearest even, the clamp makes it saturate).
#pragma once
#include "gc_internal.h"

namespace gc {
namespace {


typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }
// Saturate to the largest E4M3 magnitude; NaN stays NaN (and converts to a NaN code).
__device__ __forceinline__ float clamp448(float x) {
    return __builtin_isnan(x) ? x : fminf(fmaxf(x, -448.f), 448.f);
}

// Four bf16 values (two words) as four E4M3 codes (one word, first value lowest).
__device__ __forceinline__ uint32_t quantise4(uint32_t w0, uint32_t w1, float inv) {
    int r = __builtin_amdgcn_cvt_pk_fp8_f32(clamp448(bf16_lo(w0) * inv), clamp448(bf16_hi(w0) * inv), 0, false);
    r = __builtin_amdgcn_cvt_pk_fp8_f32(clamp448(bf16_lo(w1) * inv), clamp448(bf16_hi(w1) * inv), r, true);
    return (uint32_t)r;
}
__device__ __forceinline__ uint8_t quantise1(uint16_t x, float inv) {
    const float v = clamp448(__uint_as_float((uint32_t)x << 16) * inv);
    return (uint8_t)(__builtin_amdgcn_cvt_pk_fp8_f32(v, v, 0, false) & 0xFF);
}

// One append workgroup: tokens 16 bx .. 16 bx + 15, KV head `h`.
template <int D, bool FP8>
__device__ __forceinline__ void append_body(const AppendArgs& a, int bx, int h) {
    constexpr int CPR = D / 8;        // 16-byte chunks per row
    constexpr int kStride = D + 8;    // padded LDS row (elements)
    __shared__ int32_t s_blk[kAppendTokens];
    __shared__ int32_t s_off[kAppendTokens];
    __shared__ __align__(16) uint16_t s_v[kAppendTokens * kStride];

    const int tid = threadIdx.x;
    const int tok0 = bx * kAppendTokens;
    const int ntok = min(kAppendTokens, a.total_tokens - tok0);

    if (tid < kAppendTokens) {
        int blk = -1, off = 0;
        const int tok = tok0 + tid;
        if (tid < ntok) {
            // largest r with cu[r] <= tok; empty requests are skipped over
            int lo = 0, hi = a.batch;
            while (hi - lo > 1) {
                const int mid = (lo + hi) >> 1;
                if (a.cu_new_lens[mid] <= tok) lo = mid;
                else hi = mid;
            }
            const int pos = a.prefix_lens[lo] + (tok - a.cu_new_lens[lo]);
            const int lp = pos / kPage;
            off = pos % kPage;
            if (lp < a.max_blocks) {
                const int b = a.block_tables[(int64_t)lo * a.max_blocks + lp];
                if (b >= 0 && b < a.num_blocks) blk = b;
            }
        }
        s_blk[tid] = blk;
        s_off[tid] = off;
    }
    __syncthreads();

    for (int x = tid; x < kAppendTokens * CPR; x += kAppendThreads) {
        const int tl = x / CPR, ch = x % CPR;
        u32x4 v = u32x4{0u, 0u, 0u, 0u};
        if (tl < ntok) {
            const int64_t src = ((int64_t)(tok0 + tl) * a.num_kv_heads + h) * D + ch * 8;
            const int blk = s_blk[tl];
            if (blk >= 0) {
                const u32x4 k = *reinterpret_cast<const u32x4*>(a.k_new + src);
                const int64_t dst = (((int64_t)blk * a.num_kv_heads + h) * kPage + s_off[tl]) * D + ch * 8;
                if constexpr (FP8)
                    *reinterpret_cast<u32x2*>(static_cast<uint8_t*>(a.k_pool) + dst) =
                        u32x2{quantise4(k[0], k[1], a.k_inv), quantise4(k[2], k[3], a.k_inv)};
                else
                    *reinterpret_cast<u32x4*>(static_cast<uint16_t*>(a.k_pool) + dst) = k;
            }
            v = *reinterpret_cast<const u32x4*>(a.v_new + src);
        }
        *reinterpret_cast<u32x4*>(&s_v[tl * kStride + ch * 8]) = v;
    }
    __syncthreads();
    for (int x = tid; x < kAppendTokens * D; x += kAppendThreads) {
        const int tl = x % kAppendTokens, d = x / kAppendTokens;
        const int blk = s_blk[tl];
        if (tl < ntok && blk >= 0) {
            const int64_t dst = (((int64_t)blk * a.num_kv_heads + h) * D + d) * kPage + s_off[tl];
            if constexpr (FP8)
                static_cast<uint8_t*>(a.v_pool)[dst] = quantise1(s_v[tl * kStride + d], a.v_inv);
            else
                static_cast<uint16_t*>(a.v_pool)[dst] = s_v[tl * kStride + d];
        }
    }
}

}  // namespace
}  // namespace gc
