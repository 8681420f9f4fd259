// Small-tile attention for gfx950: the decode-like case where every request
// has only a few new tokens (GreenCache §2.1-2.2: a cached context followed by
// token-by-token generation still attends over the whole stored KV).
//
// Computes exactly what the prefill path computes (causal scaled-dot-product
// attention of the new tokens over cached prefix plus new tokens, GQA), for
// query tiles of 16 rows (the g query heads of one KV head over 16/g new
// tokens) and key tiles of 32 keys (two pool pages). Such work is bound by
// reading K and V, so each wavefront owns one work item and reads its K and V
// fragments straight from global memory into registers in the matrix-core
// operand layouts (no LDS staging, no barriers), with the next two tiles' loads
// in flight while the current tile is computed:
//   S^T (32 keys x 16 rows)  = K . Q^T     two 16x16 blocks, MFMA 16x16x32 bf16
//   O^T (D x 16 rows)       += V^T . P^T   D/16 blocks,     MFMA 16x16x32 bf16
// Score block b covers page b of the tile; the k order of the PV product is
// permuted to match, so the score accumulators are already laid out as the P^T
// operand and every global load reads a single page.
// With 8-bit pools (E4M3 codes times one scale per pool) the same fragments are
// loaded at half the width and widened to bf16 in registers (exact: every E4M3
// value is a bf16 value); the key scale is folded into the softmax scale and the
// value scale into the final normalisation, so the loop is otherwise unchanged.
#include "gc_internal.h"

namespace gc {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef const __attribute__((address_space(4))) int32_t* scalar_i32p;

constexpr float kLn2 = 0.69314718055994530942f;
// Buffer resource word 3 for raw (untyped) loads: 32-bit data format.
constexpr int kBufferFlags = 0x00020000;

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    const bf16x2 p = {(__bf16)lo, (__bf16)hi};
    return __builtin_bit_cast(uint32_t, p);
}

// x combined with the value of lane l ^ 16 (max or sum), then with lane l ^ 32
__device__ __forceinline__ float row_max4(float x) {
    const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    x = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
    const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float row_sum4(float x) {
    const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    x = __uint_as_float(a[0]) + __uint_as_float(a[1]);
    const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// Four E4M3 codes (one 32-bit word) as four bf16 values (two 32-bit words).
__device__ __forceinline__ u32x2 widen_e4m3x4(uint32_t w) {
    const bf16x2 lo = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w, 1.0f, false);
    const bf16x2 hi = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w, 1.0f, true);
    return u32x2{__builtin_bit_cast(uint32_t, lo), __builtin_bit_cast(uint32_t, hi)};
}

// Register fragments of one key tile: K^T operands per (page, k-step) and four
// value slots per (page, value block), at the pool's element width.
template <int D, bool FP8>
struct SmallFrags;
template <int D>
struct SmallFrags<D, false> {
    bf16x8 k[2][D / 32];
    u32x2 v[2][D / 16];
    __device__ __forceinline__ bf16x8 kop(int b, int s) const { return k[b][s]; }
    __device__ __forceinline__ u32x2 vop(int b, int db) const { return v[b][db]; }
};
template <int D>
struct SmallFrags<D, true> {
    u32x4 k[2][D / 64];      // 16 codes: the K^T operands of k-steps 2p and 2p + 1
    uint32_t v[2][D / 16];   // 4 codes
    __device__ __forceinline__ bf16x8 kop(int b, int s) const {
        const u32x4 w = k[b][s >> 1];
        const u32x2 a = widen_e4m3x4(w[2 * (s & 1)]), c = widen_e4m3x4(w[2 * (s & 1) + 1]);
        return __builtin_bit_cast(bf16x8, u32x4{a[0], a[1], c[0], c[1]});
    }
    __device__ __forceinline__ u32x2 vop(int b, int db) const { return widen_e4m3x4(v[b][db]); }
};

template <int D, bool FP8>
__global__ __launch_bounds__(kDecWaves * 64, 1) void attention_small_kernel(const AttnArgs a, int64_t units) {
    constexpr int KS = D / 32;                    // k-steps of QK^T
    constexpr int DB = D / 16;                    // 16-row blocks of O^T
    constexpr int kTileLog2Thresh = 8;            // rescale only when the max grows by > 2^8
    static_assert(kDecM == 16 && kDecN == 32 && kPage == 16, "tile shape");

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    const int64_t u = (int64_t)blockIdx.x * kDecWaves + wave;
    if (u >= units) return;
    const int kvh = (int)(u % a.num_kv_heads);
    const WorkItem it = a.items[u / a.num_kv_heads];
    if (it.r < 0 || it.kt_begin >= it.kt_end) return;

    const int r = it.r;
    const int P = a.prefix_lens[r];
    const int cu = a.cu_new_lens[r];
    const int n = a.cu_new_lens[r + 1] - cu;
    const int L = P + n;
    const int ntok = min(a.tq, n - it.q0);

    const int g4 = lane >> 4;   // lane group: keys 8 g4 .. 8 g4 + 7 of a tile
    const int j = lane & 15;    // query row of the tile: token t, head kvh * g + hl
    const int t = j / a.group;
    const int hl = j - t * a.group;
    const bool row_ok = t < ntok;
    const int lim = P + it.q0 + (row_ok ? t : 0);  // last key this row may see
    const int64_t qrow = (int64_t)(cu + it.q0 + t) * a.num_q_heads + kvh * a.group + hl;

    // Q^T operand of k-step s: lane holds q[row j][32 s + 8 g4 .. +7]. Over 8-bit
    // pools the head dimension is taken in another order (the sum over d does not
    // depend on it): k-steps 2p and 2p + 1 cover d = 64 p + 16 g4 .. +15 of lane
    // group g4, so one 16-byte load brings a lane's K codes for both steps.
    bf16x8 qf[KS];
#pragma unroll
    for (int s = 0; s < KS; ++s) {
        const int d0 = FP8 ? 64 * (s >> 1) + 16 * g4 + 8 * (s & 1) : 32 * s + 8 * g4;
        qf[s] = row_ok ? *reinterpret_cast<const bf16x8*>(a.q + qrow * D + d0)
                       : __builtin_bit_cast(bf16x8, u32x4{0u, 0u, 0u, 0u});
    }

    // Score block b holds the 16 keys of page b of the tile (operand row i = key
    // slot i), so accumulator value v of block b is key 16 b + 4 g4 + v. The P^T
    // operand takes value (b, v) as its k index 8 g4 + 4 b + v; the V^T operand
    // uses the same key order: lane (d, g4) holds slots 4 g4 .. 4 g4 + 3 of both
    // pages. Every load reads one page, at a wave-uniform page address plus a
    // per-lane offset.
    const scalar_i32p table = (scalar_i32p)(a.block_tables + (int64_t)r * a.max_blocks);
    constexpr int EB = FP8 ? 1 : 2;  // bytes per pool element
    const int64_t page_bytes = (int64_t)kPage * D * EB;
    const int64_t block_bytes = (int64_t)a.num_kv_heads * page_bytes;
    const unsigned char* kbase = reinterpret_cast<const unsigned char*>(a.k_pool) + (int64_t)kvh * page_bytes;
    const unsigned char* vbase = reinterpret_cast<const unsigned char*>(a.v_pool) + (int64_t)kvh * page_bytes;
    const uint32_t k_off = (uint32_t)(j * D + (FP8 ? 16 : 8) * g4) * EB;  // + 64 B per k-step (pair)
    const uint32_t v_off = (uint32_t)(j * kPage + 4 * g4) * EB;     // + 256 EB db bytes per value block

    using Frags = SmallFrags<D, FP8>;
    // Block ids of the two pages of tile kt (scalar loads, fetched a tile ahead of
    // their use); pages past the sequence end or with an out-of-range id read
    // block 0 instead (their keys are masked, values zeroed).
    struct Ids {
        int b0, b1;
    };
    auto fetch_ids = [&](int kt) -> Ids {
        return Ids{table[min(kt * 2, a.max_blocks - 1)], table[min(kt * 2 + 1, a.max_blocks - 1)]};
    };
    auto page_block = [&](int kt, int p, int blk) -> int64_t {
        const int lp = kt * 2 + p;
        const bool ok = (lp < a.max_blocks) & (lp * kPage < L) & (blk >= 0) & (blk < a.num_blocks);
        return ok ? blk : 0;
    };
    // Loads go through buffer resources (one per page, in scalar registers) with
    // loop-invariant per-lane offsets, so a tile's loads need no address registers
    // that could collide with fragments still in flight. A page resource covers
    // exactly the page; nothing outside it can be read.
    auto load = [&](int kt, const Ids& ids, Frags& f) {
        const int64_t blk[2] = {page_block(kt, 0, ids.b0), page_block(kt, 1, ids.b1)};
#pragma unroll
        for (int b = 0; b < 2; ++b) {
            const __amdgpu_buffer_rsrc_t kr = __builtin_amdgcn_make_buffer_rsrc(
                (void*)(kbase + blk[b] * block_bytes), (short)0, (int)page_bytes, kBufferFlags);
            const __amdgpu_buffer_rsrc_t vr = __builtin_amdgcn_make_buffer_rsrc(
                (void*)(vbase + blk[b] * block_bytes), (short)0, (int)page_bytes, kBufferFlags);
            if constexpr (FP8) {
#pragma unroll
                for (int p = 0; p < KS / 2; ++p)
                    f.k[b][p] = __builtin_amdgcn_raw_buffer_load_b128(kr, (int)k_off + 64 * p, 0, 0);
#pragma unroll
                for (int db = 0; db < DB; ++db)
                    f.v[b][db] = __builtin_amdgcn_raw_buffer_load_b32(vr, (int)v_off + 256 * db, 0, 0);
            } else {
#pragma unroll
                for (int s = 0; s < KS; ++s)
                    f.k[b][s] = __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(kr, (int)k_off + 64 * s, 0, 0));
#pragma unroll
                for (int db = 0; db < DB; ++db)
                    f.v[b][db] = __builtin_amdgcn_raw_buffer_load_b64(vr, (int)v_off + 512 * db, 0, 0);
            }
        }
    };

    f32x4 o[DB];
#pragma unroll
    for (int db = 0; db < DB; ++db) o[db] = f32x4{0.f, 0.f, 0.f, 0.f};
    float m_run = -INFINITY;  // exponent offset in score * scale * log2(e) units
    float l_run = 0.f;        // this lane's share of the row sum of the bf16 weights
    const float c = a.scale_log2;
    const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};

    auto compute = [&](int kt, Frags& f) {
        f32x4 s[2];
#pragma unroll
        for (int b = 0; b < 2; ++b) {
            s[b] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int ks = 0; ks < KS; ++ks)
                s[b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(f.kop(b, ks), qf[ks], s[b], 0, 0, 0);
        }
        // value fragments as bf16 words (widened here for 8-bit pools)
        u32x2 vw[2][DB];
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
            for (int db = 0; db < DB; ++db) vw[b][db] = f.vop(b, db);
        // s[b][v] is the score of tile key 16 b + 4 g4 + v
        const int key0 = kt * kDecN;
        if (key0 + kDecN - 1 > P + it.q0) {
            const int rel = lim - key0 - 4 * g4;
#pragma unroll
            for (int b = 0; b < 2; ++b)
#pragma unroll
                for (int v = 0; v < 4; ++v) s[b][v] = (16 * b + v > rel) ? -INFINITY : s[b][v];
            // values past the sequence end become 0 (weight 0 times a stale value)
            const int bad = L - key0 - 4 * g4;  // first of this lane's slots (16 b + v) at or past the end
            if (bad < 20) {
#pragma unroll
                for (int b = 0; b < 2; ++b)
#pragma unroll
                    for (int db = 0; db < DB; ++db)
#pragma unroll
                        for (int x = 0; x < 2; ++x)
                            vw[b][db][x] &= (16 * b + 2 * x < bad ? 0xFFFFu : 0u) |
                                            (16 * b + 2 * x + 1 < bad ? 0xFFFF0000u : 0u);
            }
        }
        float mx = fmaxf(fmaxf(fmaxf(s[0][0], s[0][1]), fmaxf(s[0][2], s[0][3])),
                         fmaxf(fmaxf(s[1][0], s[1][1]), fmaxf(s[1][2], s[1][3])));
        const float m_tile = row_max4(mx) * c;
        if (__any(m_tile > m_run + kTileLog2Thresh)) {
            const float m_new = fmaxf(m_run, m_tile);
            // rows that have seen no visible key yet keep o = l = 0 with any finite alpha
            const float alpha = m_new == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m_run - m_new);
            m_run = m_new;
            l_run *= alpha;
#pragma unroll
            for (int db = 0; db < DB; ++db) o[db] *= alpha;
        }
        const float m_use = (m_run == -INFINITY) ? 0.f : m_run;
        u32x4 pw;
#pragma unroll
        for (int x = 0; x < 4; ++x) {
            const float p0 = __builtin_amdgcn_exp2f(fmaf(s[x >> 1][2 * (x & 1)], c, -m_use));
            const float p1 = __builtin_amdgcn_exp2f(fmaf(s[x >> 1][2 * (x & 1) + 1], c, -m_use));
            const bf16x2 pair = {(__bf16)p0, (__bf16)p1};
            l_run = __builtin_amdgcn_fdot2_f32_bf16(pair, ones, l_run, false);
            pw[x] = __builtin_bit_cast(uint32_t, pair);
        }
        const bf16x8 pf = __builtin_bit_cast(bf16x8, pw);
#pragma unroll
        for (int db = 0; db < DB; ++db) {
            const u32x4 vv = {vw[0][db][0], vw[0][db][1], vw[1][db][0], vw[1][db][1]};
            o[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, vv), pf, o[db], 0, 0, 0);
        }
    };

    // NS fragment sets used in turn (no register copies): the loads of tiles kt+1 ..
    // kt+NS-1 are in flight while tile kt is computed. Loads are issued
    // unconditionally (past the last tile the last tile is loaded again), so the
    // compiler's wait before a tile's products covers exactly that tile's loads.
    // 8-bit tiles take 20 loads per lane, so three tiles ahead stay within the
    // 63 loads the vector-memory counter can track; bf16 tiles (24 loads, twice
    // the registers) keep two.
    constexpr int NS = FP8 ? 4 : 3;
    Frags f0, f1, f2, f3;
    const int kt_end = it.kt_end, last = kt_end - 1;
    int kt = it.kt_begin;
    load(kt, fetch_ids(kt), f0);
    load(min(kt + 1, last), fetch_ids(min(kt + 1, last)), f1);
    if constexpr (NS == 4) load(min(kt + 2, last), fetch_ids(min(kt + 2, last)), f2);
    Ids ids = fetch_ids(min(kt + NS - 1, last));
    auto step = [&](Frags& cur, Frags& ahead) {
        load(min(kt + NS - 1, last), ids, ahead);
        ids = fetch_ids(min(kt + NS, last));
        compute(kt, cur);
    };
    if constexpr (NS == 3) {
        while (true) {
            step(f0, f2);
            if (++kt >= kt_end) break;
            step(f1, f0);
            if (++kt >= kt_end) break;
            step(f2, f1);
            if (++kt >= kt_end) break;
        }
    } else {
        while (true) {
            step(f0, f3);
            if (++kt >= kt_end) break;
            step(f1, f0);
            if (++kt >= kt_end) break;
            step(f2, f1);
            if (++kt >= kt_end) break;
            step(f3, f2);
            if (++kt >= kt_end) break;
        }
    }

    const float l_tot = row_sum4(l_run);
    const float inv = l_tot > 0.f ? a.v_scale / l_tot : 0.f;  // v_scale is 1 for bf16 pools
    const float lse_v = l_tot > 0.f ? (m_run + log2f(l_tot)) * kLn2 : -INFINITY;
    // o[db][v] is element d = 16 db + 4 g4 + v of row j
    if (it.part < 0) {
        if (row_ok) {
            uint16_t* op = a.out + qrow * D + 4 * g4;
#pragma unroll
            for (int db = 0; db < DB; ++db) {
                u32x2 w;
                w[0] = pack_bf16x2(o[db][0] * inv, o[db][1] * inv);
                w[1] = pack_bf16x2(o[db][2] * inv, o[db][3] * inv);
                *reinterpret_cast<u32x2*>(op + 16 * db) = w;
            }
            if (a.lse != nullptr && g4 == 0) a.lse[qrow] = lse_v;
        }
    } else {
        const int64_t prow = ((int64_t)it.part * a.num_kv_heads + kvh) * kDecM + j;
        float* po = a.part_o + prow * D + 4 * g4;
#pragma unroll
        for (int db = 0; db < DB; ++db) *reinterpret_cast<f32x4*>(po + 16 * db) = o[db] * inv;
        if (g4 == 0) a.part_lse[prow] = lse_v;
    }
}

}  // namespace

hipError_t launch_attention_small(const AttnArgs& a, int head_dim, int64_t num_items, bool fp8,
                                  hipStream_t s) {
    const int64_t units = num_items * a.num_kv_heads;
    const dim3 grid((unsigned)ceil_div64(units, kDecWaves));
    if (fp8) {
        if (head_dim == 128)
            attention_small_kernel<128, true><<<grid, kDecWaves * 64, 0, s>>>(a, units);
        else
            attention_small_kernel<64, true><<<grid, kDecWaves * 64, 0, s>>>(a, units);
    } else {
        if (head_dim == 128)
            attention_small_kernel<128, false><<<grid, kDecWaves * 64, 0, s>>>(a, units);
        else
            attention_small_kernel<64, false><<<grid, kDecWaves * 64, 0, s>>>(a, units);
    }
    return hipGetLastError();
}

}  // namespace gc
