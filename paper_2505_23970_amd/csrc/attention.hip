// Prefix-cached prefill attention and split-KV merge for gfx950 (CDNA4).
//
// Computes, for every new token of every request and every query head, causal
// scaled-dot-product attention over the request's cached prefix keys plus the
// new keys up to and including the token itself (GreenCache §2.2, Fig. 1a:
// cached and new KV processed together; §2.1 prefill). Keys are gathered from
// the paged pool through the block table.
//
// Work decomposition. A workgroup (4 wavefronts) owns one work item: 128 query
// rows = the g query heads of one KV head stacked over 128/g consecutive new
// tokens of one request, against a range of 64-key tiles. Each wavefront owns
// 32 of the rows. Per key tile:
//   S^T (64 keys x 32 rows)  = K_tile . Q^T        two 32x32 blocks, MFMA 32x32x16 bf16
//   online softmax on S^T in registers               fp32, base-2 exponent
//   O^T (D x 32 rows)       += V_tile^T . P^T       D/32 blocks, MFMA 32x32x16 bf16
// Computing the transposed products puts every score of one query row in one
// lane pair (lanes l and l+32), so row maxima and sums are in-lane plus one
// cross-half exchange, and the QK^T accumulator doubles as the PV operand
// once the key rows fed to the first product are permuted (bits 2 and 3 of
// the row index swapped).
// K and V tiles are staged through LDS, double buffered: the next tile's
// global loads are in flight while the current tile is computed. Value pages
// are stored transposed in the pool ([D][16]), so both LDS tiles are read with
// 16-byte loads; XOR swizzles keep those reads free of bank conflicts.
#include "gc_internal.h"

namespace gc {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr float kLn2 = 0.69314718055994530942f;

// 16-byte chunk position inside an LDS row (conflict-free 16-lane reads).
template <int D>
__device__ __forceinline__ int swz_k(int chunk, int row) {
    if constexpr (D == 128) return chunk ^ (row & 15);  // 256-byte rows
    else return chunk ^ ((row >> 1) & 7);                // 128-byte rows
}
__device__ __forceinline__ int swz_v(int chunk, int drow) { return chunk ^ ((drow >> 1) & 7); }

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    __bf16 a = (__bf16)lo;
    __bf16 b = (__bf16)hi;
    return (uint32_t)__builtin_bit_cast(uint16_t, a) | ((uint32_t)__builtin_bit_cast(uint16_t, b) << 16);
}

template <int D>
__global__ __launch_bounds__(kAttnThreads, 2) void attention_kernel(const AttnArgs a) {
    constexpr int DK = D / 16;               // k-steps of QK^T
    constexpr int DB = D / 32;               // 32-row blocks of O^T
    constexpr int NCH = D / 32;              // 16-byte chunks per thread per tile per tensor
    constexpr int kPagesPerPass = kAttnThreads / (2 * D);

    __shared__ __align__(16) uint16_t k_lds[2][kBlockN * D];
    __shared__ __align__(16) uint16_t v_lds[2][D * kBlockN];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int hh = lane >> 5;
    const int lr = lane & 31;
    const int kvh = (int)(blockIdx.x % (unsigned)a.num_kv_heads);
    const WorkItem it = a.items[blockIdx.x / (unsigned)a.num_kv_heads];
    if (it.r < 0 || it.kt_begin >= it.kt_end) return;

    const int r = it.r;
    const int P = a.prefix_lens[r];
    const int cu = a.cu_new_lens[r];
    const int n = a.cu_new_lens[r + 1] - cu;
    const int L = P + n;
    const int ntok = min(a.tq, n - it.q0);

    // this lane's query row: token t of the tile, query head kvh * g + hl
    const int m = wave * kRowsPerWave + lr;
    const int t = m / a.group;
    const int hl = m - t * a.group;
    const bool row_ok = t < ntok;
    const int lim = P + it.q0 + (row_ok ? t : 0);  // last key this row may see
    const int64_t qrow = (int64_t)(cu + it.q0 + t) * a.num_q_heads + kvh * a.group + hl;

    // Q^T operand: lane holds q[row][16k + 8*hh .. +7]
    bf16x8 qf[DK];
    if (row_ok) {
        const uint16_t* qp = a.q + qrow * D + hh * 8;
#pragma unroll
        for (int k = 0; k < DK; ++k) qf[k] = *reinterpret_cast<const bf16x8*>(qp + 16 * k);
    } else {
#pragma unroll
        for (int k = 0; k < DK; ++k) qf[k] = __builtin_bit_cast(bf16x8, u32x4{0u, 0u, 0u, 0u});
    }

    // staging assignment: page (e * kPagesPerPass + pip) of the tile
    const int pip = tid / (2 * D);
    const int idx = tid % (2 * D);
    const int k_slot = idx / (D / 8), k_chunk = idx % (D / 8);
    const int v_row = idx >> 1, v_half = idx & 1;
    u32x4 kreg[NCH], vreg[NCH];

    auto load_tile = [&](int kt) {
#pragma unroll
        for (int e = 0; e < NCH; ++e) {
            const int p = e * kPagesPerPass + pip;
            const int lp = kt * (kBlockN / kPage) + p;
            int blk = -1;
            if (lp * kPage < L && lp < a.max_blocks) {
                blk = a.block_tables[(int64_t)r * a.max_blocks + lp];
                if (blk >= a.num_blocks) blk = -1;
            }
            if (blk >= 0) {
                const int64_t base = ((int64_t)blk * a.num_kv_heads + kvh) * (kPage * D);
                kreg[e] = *reinterpret_cast<const u32x4*>(a.k_pool + base + k_slot * D + k_chunk * 8);
                u32x4 v = *reinterpret_cast<const u32x4*>(a.v_pool + base + v_row * kPage + v_half * 8);
                const int j0 = lp * kPage + v_half * 8;
                if (j0 + 8 > L) {  // value slots at or past the sequence end become 0
#pragma unroll
                    for (int w = 0; w < 4; ++w) {
                        uint32_t keep = (j0 + 2 * w < L ? 0x0000FFFFu : 0u) |
                                        (j0 + 2 * w + 1 < L ? 0xFFFF0000u : 0u);
                        v[w] &= keep;
                    }
                }
                vreg[e] = v;
            } else {
                kreg[e] = u32x4{0u, 0u, 0u, 0u};
                vreg[e] = u32x4{0u, 0u, 0u, 0u};
            }
        }
    };
    auto store_tile = [&](int buf) {
#pragma unroll
        for (int e = 0; e < NCH; ++e) {
            const int p = e * kPagesPerPass + pip;
            const int krow = p * kPage + k_slot;
            *reinterpret_cast<u32x4*>(&k_lds[buf][krow * D + swz_k<D>(k_chunk, krow) * 8]) = kreg[e];
            *reinterpret_cast<u32x4*>(&v_lds[buf][v_row * kBlockN + swz_v(2 * p + v_half, v_row) * 8]) = vreg[e];
        }
    };

    f32x16 o[DB];
#pragma unroll
    for (int db = 0; db < DB; ++db) o[db] = f32x16{};
    float m_run = -INFINITY;  // running row max of score * scale * log2(e)
    float l_run = 0.f;        // this lane's half of the running row sum
    const float c = a.scale_log2;
    // key row fed to the QK^T product by this lane: bits 2 and 3 of lr swapped
    const int prow = (lr & 0x13) | ((lr & 4) << 1) | ((lr & 8) >> 1);

    int kt = it.kt_begin;
    load_tile(kt);
    store_tile(0);
    __syncthreads();
    for (int i = 0; kt < it.kt_end; ++kt, ++i) {
        const int buf = i & 1;
        const bool more = kt + 1 < it.kt_end;
        if (more) load_tile(kt + 1);
        const uint16_t* kb = k_lds[buf];
        const uint16_t* vb = v_lds[buf];

        f32x16 s[2];
#pragma unroll
        for (int b = 0; b < 2; ++b) {
            s[b] = f32x16{};
            const int krow = 32 * b + prow;
#pragma unroll
            for (int k = 0; k < DK; ++k) {
                const bf16x8 kf = *reinterpret_cast<const bf16x8*>(kb + krow * D + swz_k<D>(2 * k + hh, krow) * 8);
                s[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[k], s[b], 0, 0, 0);
            }
        }
        // s[b][e] is the score of key tile_base + 32b + 16(e>>3) + 8hh + (e&7)
        const int key0 = kt * kBlockN;
        if (key0 + kBlockN - 1 > P + it.q0) {
#pragma unroll
            for (int b = 0; b < 2; ++b)
#pragma unroll
                for (int e = 0; e < 16; ++e) {
                    const int key = key0 + 32 * b + 16 * (e >> 3) + 8 * hh + (e & 7);
                    if (key > lim) s[b][e] = -INFINITY;
                }
        }
        float mx = -INFINITY;
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
            for (int e = 0; e < 16; ++e) mx = fmaxf(mx, s[b][e]);
        mx = fmaxf(mx, __shfl_xor(mx, 32));
        const float m_new = fmaxf(m_run, mx * c);
        const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
        const float alpha = __builtin_amdgcn_exp2f(m_run - m_use);
        m_run = m_new;
        l_run *= alpha;
#pragma unroll
        for (int db = 0; db < DB; ++db) o[db] *= alpha;

        bf16x8 pf[4];
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const float p = __builtin_amdgcn_exp2f(fmaf(s[b][e], c, -m_use));
                l_run += p;
                pf[2 * b + (e >> 3)][e & 7] = (__bf16)p;
            }
#pragma unroll
        for (int st = 0; st < 4; ++st)
#pragma unroll
            for (int db = 0; db < DB; ++db) {
                const int d = 32 * db + lr;
                const bf16x8 vf = *reinterpret_cast<const bf16x8*>(vb + d * kBlockN + swz_v(2 * st + hh, d) * 8);
                o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[st], o[db], 0, 0, 0);
            }
        if (more) store_tile(buf ^ 1);
        __syncthreads();
    }

    const float l_tot = l_run + __shfl_xor(l_run, 32);
    const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
    const float lse_v = l_tot > 0.f ? (m_run + log2f(l_tot)) * kLn2 : -INFINITY;
    // o[db][4j + i] is element d = 32db + 8j + 4hh + i of this lane's row
    if (it.part < 0) {
        if (row_ok) {
            uint16_t* op = a.out + qrow * D;
#pragma unroll
            for (int db = 0; db < DB; ++db)
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    u32x2 w;
                    w[0] = pack_bf16x2(o[db][4 * j] * inv, o[db][4 * j + 1] * inv);
                    w[1] = pack_bf16x2(o[db][4 * j + 2] * inv, o[db][4 * j + 3] * inv);
                    *reinterpret_cast<u32x2*>(op + 32 * db + 8 * j + 4 * hh) = w;
                }
            if (a.lse != nullptr && hh == 0) a.lse[qrow] = lse_v;
        }
    } else {
        const int64_t prow_g = ((int64_t)it.part * a.num_kv_heads + kvh) * kBlockM + m;
        float* po = a.part_o + prow_g * D;
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                f32x4 w = {o[db][4 * j] * inv, o[db][4 * j + 1] * inv, o[db][4 * j + 2] * inv,
                           o[db][4 * j + 3] * inv};
                *reinterpret_cast<f32x4*>(po + 32 * db + 8 * j + 4 * hh) = w;
            }
        if (hh == 0) a.part_lse[prow_g] = lse_v;
    }
}

// Merge the key chunks of one split query tile: lse = log sum_s exp(lse_s),
// o = sum_s exp(lse_s - lse) o_s, in a fixed chunk order (deterministic).
template <int D>
__global__ __launch_bounds__(256) void combine_kernel(const CombineArgs a) {
    constexpr int CPR = D / 4;  // float4 chunks per row
    const int kvh = (int)(blockIdx.x % (unsigned)a.num_kv_heads);
    const CombineItem ci = a.combines[blockIdx.x / (unsigned)a.num_kv_heads];
    if (ci.ns <= 0) return;
    const int cu = a.cu_new_lens[ci.r];
    const int n = a.cu_new_lens[ci.r + 1] - cu;
    const int ntok = min(a.tq, n - ci.q0);
    const int rows = ntok * a.group;
    for (int x = threadIdx.x; x < rows * CPR; x += blockDim.x) {
        const int m = x / CPR, c4 = x % CPR;
        const int t = m / a.group, hl = m - t * a.group;
        float mx = -INFINITY;
        for (int s = 0; s < ci.ns; ++s)
            mx = fmaxf(mx, a.part_lse[((int64_t)(ci.part_base + s) * a.num_kv_heads + kvh) * kBlockM + m]);
        float tot = 0.f;
        for (int s = 0; s < ci.ns; ++s)
            tot += expf(a.part_lse[((int64_t)(ci.part_base + s) * a.num_kv_heads + kvh) * kBlockM + m] - mx);
        const float lse_tot = mx + logf(tot);
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
        for (int s = 0; s < ci.ns; ++s) {
            const int64_t pr = ((int64_t)(ci.part_base + s) * a.num_kv_heads + kvh) * kBlockM + m;
            const float w = expf(a.part_lse[pr] - lse_tot);
            const f32x4 v = *reinterpret_cast<const f32x4*>(a.part_o + pr * D + 4 * c4);
            acc += w * v;
        }
        const int64_t qrow = (int64_t)(cu + ci.q0 + t) * a.num_q_heads + kvh * a.group + hl;
        u32x2 w2;
        w2[0] = pack_bf16x2(acc[0], acc[1]);
        w2[1] = pack_bf16x2(acc[2], acc[3]);
        *reinterpret_cast<u32x2*>(a.out + qrow * D + 4 * c4) = w2;
        if (a.lse != nullptr && c4 == 0) a.lse[qrow] = lse_tot;
    }
}

}  // namespace

hipError_t launch_attention(const AttnArgs& a, int head_dim, int64_t num_items, hipStream_t s) {
    const dim3 grid((unsigned)(num_items * a.num_kv_heads));
    if (head_dim == 128)
        attention_kernel<128><<<grid, kAttnThreads, 0, s>>>(a);
    else
        attention_kernel<64><<<grid, kAttnThreads, 0, s>>>(a);
    return hipGetLastError();
}

hipError_t launch_combine(const CombineArgs& a, int head_dim, int64_t num_combines, hipStream_t s) {
    const dim3 grid((unsigned)(num_combines * a.num_kv_heads));
    if (head_dim == 128)
        combine_kernel<128><<<grid, 256, 0, s>>>(a);
    else
        combine_kernel<64><<<grid, 256, 0, s>>>(a);
    return hipGetLastError();
}

}  // namespace gc
