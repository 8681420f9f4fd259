// KV append for gfx950 (device code shared by the append kernel and the fused
// append-and-plan launch): copy the new tokens' K/V into their pool slots
// (GreenCache §2.2, Fig. 1a step 1: the processed request's KV is saved so a
// later request with the same context can reuse it).
//
// A workgroup owns one destination page of one KV head: (request r, logical
// page lp, head h) for every page that receives at least one new token, i.e.
// pages P_r / 16 .. (P_r + n_r - 1) / 16 of every request. The pages of the
// whole batch are numbered request by request; a workgroup finds its request
// with a block-wide scan of the per-request page counts (one pass for batches
// of up to 256 requests). The page's new slots [s0, s1) are contiguous:
//   - keys: each slot's row is D contiguous elements in the page, copied in
//     16-byte chunks (one chunk per thread);
//   - values: the page is stored transposed ([D][16] slots), so the tokens'
//     rows are staged in LDS and every (value row d, half of the 16 slots) is
//     written as one 16-byte store (8-byte store for 8-bit pools) when the new
//     slots cover the half, element by element where they cover part of it.
// Slots outside [s0, s1) keep their bytes (the cached prefix before P_r, and
// whatever the caller holds past the sequence end). A page whose block id is
// outside the pool, or past the table row, is skipped. If the device lengths
// disagree with the host's page count, pages beyond them are skipped and no
// token row outside [0, T) is read.
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

// Pages of request r that receive new tokens (0 for an empty request, or for
// lengths no valid batch has).
__device__ __forceinline__ int pages_receiving(int64_t P, int64_t n) {
    if (n <= 0 || P < 0) return 0;
    const int64_t p = (P + n + kPage - 1) / kPage - P / kPage;
    return p > INT32_MAX / 4 ? 0 : (int)p;
}

// LDS of one append workgroup (the caller provides it, so that a launch that
// also runs the planner can overlay the two).
template <int D>
struct AppendLds {
    static constexpr int kStride = D + 8;       // padded LDS row (elements)
    uint16_t v[kPage * kStride];                 // the page's new value rows, slot-major
    int scan[kAppendThreads / 64];               // wavefront totals of the page-count scan
    int found_r, found_k;
};

// Exclusive scan of one value per thread over the workgroup (kAppendThreads);
// *total receives the sum.
__device__ __forceinline__ int append_scan(int v, int* s_waves, int* total) {
    constexpr int kW = kAppendThreads / 64;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    int x = v;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const int y = __shfl_up(x, d);
        if (lane >= d) x += y;
    }
    if (lane == 63) s_waves[wave] = x;
    __syncthreads();
    int base = 0, tot = 0;
#pragma unroll
    for (int w = 0; w < kW; ++w) {
        const int t = s_waves[w];
        base += w < wave ? t : 0;
        tot += t;
    }
    __syncthreads();
    *total = tot;
    return base + x - v;
}

// One append workgroup: page unit u (over the batch, request-major), KV head h.
template <int D, bool FP8>
__device__ __forceinline__ void append_body(const AppendArgs& a, AppendLds<D>& sm, int u, int h) {
    constexpr int CPR = D / 8;  // 16-byte chunks per row
    constexpr int kStride = AppendLds<D>::kStride;
    const int tid = threadIdx.x;

    // 1. which request and which of its pages: scan the per-request page counts
    if (tid == 0) sm.found_r = -1;
    int carry = 0;
    for (int base = 0; base < a.batch; base += kAppendThreads) {
        const int r = base + tid;
        int pg = 0;
        if (r < a.batch) {
            const int c0 = a.cu_new_lens[r];
            pg = pages_receiving(a.prefix_lens[r], (int64_t)a.cu_new_lens[r + 1] - c0);
        }
        int total;
        const int excl = append_scan(pg, sm.scan, &total);
        if (pg > 0 && u >= carry + excl && u - (carry + excl) < pg) {
            sm.found_r = r;
            sm.found_k = u - (carry + excl);
        }
        carry += total;
        __syncthreads();
        if (sm.found_r >= 0 || carry > u) break;
    }
    const int r = sm.found_r;
    if (r < 0) return;
    const int P = a.prefix_lens[r];
    const int cu = a.cu_new_lens[r];
    const int n = a.cu_new_lens[r + 1] - cu;
    const int lp = P / kPage + sm.found_k;               // logical page
    const int s0 = max(P - lp * kPage, 0);                // first new slot of the page
    const int s1 = min(P + n - lp * kPage, kPage);        // one past the last
    if (lp >= a.max_blocks) return;
    const int blk = a.block_tables[(int64_t)r * a.max_blocks + lp];
    if (blk < 0 || blk >= a.num_blocks) return;
    // packed row of slot s: cu + lp * 16 + s - P
    const int64_t row0 = (int64_t)cu + (int64_t)lp * kPage - P;
    const int64_t page = (int64_t)blk * a.num_kv_heads + h;   // (block, head) page index

    // 2. keys straight through; values into LDS (slots outside [s0, s1) as 0, unused)
    if (tid < kPage * CPR) {
        const int s = tid / CPR, c = tid % CPR;
        const int64_t row = row0 + s;
        const bool ok = s >= s0 && s < s1 && row >= 0 && row < a.total_tokens;
        u32x4 v = u32x4{0u, 0u, 0u, 0u};
        if (ok) {
            const int64_t src = (row * a.num_kv_heads + h) * D + c * 8;
            const u32x4 k = *reinterpret_cast<const u32x4*>(a.k_new + src);
            v = *reinterpret_cast<const u32x4*>(a.v_new + src);
            const int64_t dst = (page * kPage + s) * D + c * 8;
            if constexpr (FP8)
                *reinterpret_cast<u32x2*>(static_cast<uint8_t*>(a.k_pool) + dst) =
                    u32x2{quantise4(k[0], k[1], a.k_inv), quantise4(k[2], k[3], a.k_inv)};
            else
                *reinterpret_cast<u32x4*>(static_cast<uint16_t*>(a.k_pool) + dst) = k;
        }
        *reinterpret_cast<u32x4*>(&sm.v[s * kStride + c * 8]) = v;
    }
    __syncthreads();

    // 3. values: thread (d, half) writes slots 8 half .. 8 half + 7 of value row d
    if (tid < 2 * D) {
        const int d = tid >> 1, half = tid & 1;
        const int x0 = 8 * half;
        const int64_t dst = (page * D + d) * kPage + x0;
        uint16_t e[8];
#pragma unroll
        for (int x = 0; x < 8; ++x) e[x] = sm.v[(x0 + x) * kStride + d];
        if (x0 >= s0 && x0 + 8 <= s1) {
            if constexpr (FP8) {
                const uint32_t w0 = (uint32_t)e[0] | ((uint32_t)e[1] << 16), w1 = (uint32_t)e[2] | ((uint32_t)e[3] << 16);
                const uint32_t w2 = (uint32_t)e[4] | ((uint32_t)e[5] << 16), w3 = (uint32_t)e[6] | ((uint32_t)e[7] << 16);
                *reinterpret_cast<u32x2*>(static_cast<uint8_t*>(a.v_pool) + dst) =
                    u32x2{quantise4(w0, w1, a.v_inv), quantise4(w2, w3, a.v_inv)};
            } else {
                u32x4 w;
#pragma unroll
                for (int i = 0; i < 4; ++i) w[i] = (uint32_t)e[2 * i] | ((uint32_t)e[2 * i + 1] << 16);
                *reinterpret_cast<u32x4*>(static_cast<uint16_t*>(a.v_pool) + dst) = w;
            }
        } else {
#pragma unroll
            for (int x = 0; x < 8; ++x) {
                if (x0 + x < s0 || x0 + x >= s1) continue;
                if constexpr (FP8)
                    static_cast<uint8_t*>(a.v_pool)[dst + x] = quantise1(e[x], a.v_inv);
                else
                    static_cast<uint16_t*>(a.v_pool)[dst + x] = e[x];
            }
        }
    }
}

}  // namespace
}  // namespace gc
