// Prefix-cached prefill attention and split-KV merge for gfx950 (CDNA4).
//
// Computes, for every new token of every request and every query head, causal
// scaled-dot-product attention over the request's cached prefix keys plus the
// new keys up to and including the token itself (GreenCache §2.2, Fig. 1a:
// cached and new KV processed together; §2.1 prefill). Keys are gathered from
// the paged pool through the block table.
//
// Work decomposition. A workgroup (4 wavefronts, or 8 for the wide tiling) owns
// one work item: 128 (256) query rows = the g query heads of one KV head stacked
// over consecutive new tokens of one request, against a range of 64-key tiles.
// Each wavefront owns 32 of the rows. Per key tile:
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
// The tile copies go straight from global memory to LDS; they are issued as
// inline assembly with explicit waits, so the compiler's own LDS waits count
// only LDS reads and can keep several fragment reads in flight per MFMA
// (scheduling fences hold that order).
// 8-bit pools (E4M3 codes times one scale per pool): the next tile's codes are
// loaded into registers instead, widened to bf16 (exact) and written to the same
// LDS layout after the current tile's products, so the compute loop is shared;
// the key scale is folded into the softmax scale, the value scale into the
// final normalisation.
#pragma once
#include "gc_internal.h"

namespace gc {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

constexpr float kLn2 = 0.69314718055994530942f;
// Buffer resource word 3 for raw (untyped) loads: 32-bit data format.
constexpr int kBufferFlags = 0x00020000;

// 16-byte chunk position inside an LDS row (conflict-free 16-lane reads).
template <int D>
__device__ __forceinline__ int swz_k(int chunk, int row) {
    if constexpr (D == 128) return chunk ^ (row & 15);  // 256-byte rows
    else return chunk ^ ((row >> 1) & 7);                // 128-byte rows
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    __bf16 a = (__bf16)lo;
    __bf16 b = (__bf16)hi;
    return (uint32_t)__builtin_bit_cast(uint16_t, a) | ((uint32_t)__builtin_bit_cast(uint16_t, b) << 16);
}


// A direct global->LDS copy of 16 bytes per lane: lane i's bytes land at
// lds_dst + 16 i (lds_dst is wave-uniform). Issued as inline assembly so the
// compiler does not track it: every wait for these copies is explicit (wait_vmem).
// The compiler emits no other use of m0 in these kernels; the clobber keeps it that way.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void dma16(const void* gsrc, const unsigned char* lds_dst) {
    const uint32_t l = __builtin_amdgcn_readfirstlane(
        (uint32_t)(uintptr_t)(__attribute__((address_space(3))) const unsigned char*)lds_dst);
    asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
                 :: "v"(gsrc), "s"(l) : "memory", "m0");
}
#pragma clang diagnostic pop

// Wait until at most N vector-memory operations of this wave are outstanding
// (s_waitcnt immediate: vmcnt in bits 3:0, expcnt 6:4 and lgkmcnt 11:8 left at
// their maxima). A real wait instruction, so the compiler also knows it.
template <int N>
__device__ __forceinline__ void wait_vmem() {
    static_assert(N >= 0 && N < 16, "vmcnt field");
    __builtin_amdgcn_s_waitcnt(0x0F70 | N);
    asm volatile("" ::: "memory");  // no LDS access moves above the wait
}

// The lanes of one wavefront exchange data through LDS: a release and an acquire at
// wavefront scope between the writes and the reads, so the compiler neither reuses
// values a lane loaded earlier nor moves the reads across the writes of other lanes
// (the hardware runs one wavefront's LDS operations in order).
__device__ __forceinline__ void wave_lds_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Sixteen E4M3 codes (four words) as sixteen bf16 values (eight words).
__device__ __forceinline__ void widen_e4m3x16(const u32x4 c, u32x4& lo, u32x4& hi) {
    uint32_t w[8];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        w[2 * i] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(c[i], 1.0f, false));
        w[2 * i + 1] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(c[i], 1.0f, true));
    }
    lo = u32x4{w[0], w[1], w[2], w[3]};
    hi = u32x4{w[4], w[5], w[6], w[7]};
}

// One work item (a workgroup of WAVES wavefronts): the item of launch index bid
// (blockIdx.x in the regular launch), i.e. work item bid / Hkv for KV head bid % Hkv. FUSE: the KV append runs in the
// same launch, so the keys at or past the prefix length are taken from the new
// tokens' arrays, not from the pool (bf16 pools only).
template <int D, int WAVES, bool FP8, bool FUSE>
__device__ __forceinline__ void attention_body(const AttnArgs& a, const unsigned bid) {
    static_assert(!(FP8 && FUSE), "the fused append runs over bf16 pools");
    constexpr int kBlockRows = WAVES * kRowsPerWave;  // query rows of a work item
    constexpr int DK = D / 16;                      // k-steps of QK^T
    constexpr int DB = D / 32;                      // 32-row blocks of O^T
    constexpr int kPageBytes = kPage * D * 2;       // one (block, KV head) page of K or V
    constexpr int kTileBytes = kBlockN * D * 2;     // four pages
    constexpr int kKbPerPage = kPageBytes / 1024;   // 1 KiB pieces per page
    constexpr int NI = kTileBytes / (WAVES * 1024);  // direct loads per wave per tensor per tile
    constexpr int kTileLog2Thresh = 8;              // rescale only when the max grows by > 2^8

    // K tile: [64 keys][D], row-major, 16-byte chunks XOR-swizzled by row.
    // V tile: 4 pages of [D][16 keys], the two 16-byte halves of a row swapped on odd 8-row groups.
    // Two separate buffers of each (distinct objects, so the compiler can tell that
    // reads of one do not wait for the asynchronous loads into the other).
    __shared__ __align__(16) unsigned char k_lds0[kTileBytes];
    __shared__ __align__(16) unsigned char v_lds0[kTileBytes];
    __shared__ __align__(16) unsigned char k_lds1[kTileBytes];
    __shared__ __align__(16) unsigned char v_lds1[kTileBytes];

    // (opaque to the compiler, so that the lane constants derived from it are computed per
    // work item: hoisted out of the resident launch's item loop they would be held, or
    // spilled, across the tile loop)
    int tid_opaque = (int)threadIdx.x;
    asm volatile("" : "+v"(tid_opaque));
    const int tid = tid_opaque;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int hh = lane >> 5;
    const int lr = lane & 31;
    const int kvh = (int)(bid % (unsigned)a.num_kv_heads);
    const WorkItem it = a.items[bid / (unsigned)a.num_kv_heads];
    // all eight fields in one load (else the fields the test below needs are loaded
    // first and the rest after it, a second dependent round trip)
    asm volatile("" ::"s"(it.r), "s"(it.q0), "s"(it.kt_begin), "s"(it.kt_end), "s"(it.part), "s"(it.P),
                 "s"(it.cu), "s"(it.n));
    if (it.r < 0 || it.kt_begin >= it.kt_end) return;

    // (the planner repeats the request's lengths in the item: one load for all of them)
    const int r = it.r;
    const int P = it.P;
    const int cu = it.cu;
    const int n = it.n;
    const int L = P + n;
    const int ntok = min(a.tq, n - it.q0);

    // this lane's query row: token t of the tile, query head kvh * g + hl
    const int m = wave * kRowsPerWave + lr;
    const int t = m / a.group;
    const int hl = m - t * a.group;
    const bool row_ok = t < ntok;
    const int lim = P + it.q0 + (row_ok ? t : 0);  // last key this row may see
    const int64_t qrow = (int64_t)(cu + it.q0 + t) * a.num_q_heads + kvh * a.group + hl;

    // block-table entries of the first key tile, loaded before Q: loads return in
    // order, so the first tile's copies then wait for these entries only and go out
    // while Q is still in flight (entry p in lanes with lane % 4 == p; clamped into
    // the row, checked at use)
    int ids = a.block_tables[(int64_t)r * a.max_blocks + min(it.kt_begin * 4 + (lane & 3), a.max_blocks - 1)];

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

    // Direct global->LDS loads: instruction e of a wave moves 1 KiB piece 4e + wave of
    // a tile tensor, i.e. piece `sub` of page `page_of(e)`; lane i lands at byte 16 i.
    const int sub = wave % kKbPerPage;
    static_assert(WAVES % kKbPerPage == 0, "piece layout");
    auto page_of = [&](int e) -> int { return (WAVES / kKbPerPage) * e + (wave & (WAVES - 1)) / kKbPerPage; };
    const int k_row = sub * (1024 / (2 * D)) + lane / (D / 8);         // key slot in the page
    const uint32_t k_chunk = swz_k<D>(lane % (D / 8), k_row) * 16;     // source chunk of the row
    const uint32_t k_src = k_row * (2 * D) + k_chunk;
    const int v_d = sub * 32 + (lane >> 1);                            // value row (d) in the page
    const int v_half = (lane & 1) ^ ((v_d >> 3) & 1);                  // logical half held by the lane
    const uint32_t v_src = v_d * 32 + v_half * 16;
    const int32_t* table = a.block_tables + (int64_t)r * a.max_blocks;
    const int64_t head_off = (int64_t)kvh * kPageBytes;
    const int64_t block_stride = (int64_t)a.num_kv_heads * kPageBytes;
    // fused append: this KV head's rows of the request's new tokens (new key P + i at
    // row i) and the byte stride between consecutive tokens
    const int64_t new_stride = (int64_t)a.num_kv_heads * D * 2;
    auto new_rows = [&](const uint16_t* base) {
        return reinterpret_cast<const unsigned char*>(base) + ((int64_t)cu * a.num_kv_heads + kvh) * D * 2;
    };
    const unsigned char* k_new_h = FUSE ? new_rows(a.k_new) : nullptr;
    // the values as a buffer of exactly these rows' bytes (the host keeps them < 2 GiB)
    const __amdgpu_buffer_rsrc_t v_new_r = __builtin_amdgcn_make_buffer_rsrc(
        FUSE ? (void*)new_rows(a.v_new) : nullptr, (short)0,
        FUSE ? (int)((int64_t)max(n - 1, 0) * new_stride + 2 * D) : 0, kBufferFlags);

    // raw table entries of tile kt (indices clamped into the row; checked at use)
    // (a vector load: lane p of every 4 holds entry p; it completes with the tile loads,
    // and no scalar load is left in flight to force full LDS waits in the compute phase)
    auto fetch_ids = [&](int kt, int& ids) {
        ids = table[min(kt * 4 + (lane & 3), a.max_blocks - 1)];
    };
    // Copies of piece e of tile kt (one page of K and of V for this wave). Plain
    // attention: a page past the table, past the sequence or with a block id outside
    // the pool is copied from block 0 instead (its keys are masked and its values
    // zeroed after the copy), so the copy needs no branch and can be issued between
    // the products of the tile before. Fused append: pages that are not copied are
    // skipped, and a page of new keys takes its values from registers.
    // (blk: the raw table entry of the page, read from the lanes of `ids` beforehand)
    auto issue_page = [&](unsigned char* kdst, unsigned char* vdst, int kt, const int blk, int e) {
        const int pg = page_of(e);
        const int lp = kt * 4 + pg;
        const bool ok = lp < a.max_blocks && lp * kPage < L && blk >= 0 && blk < a.num_blocks;
        const unsigned char* kpool = reinterpret_cast<const unsigned char*>(a.k_pool);
        const unsigned char* vpool = reinterpret_cast<const unsigned char*>(a.v_pool);
        if constexpr (!FUSE) {
            const int64_t base = (int64_t)(ok ? blk : 0) * block_stride + head_off;
            dma16(kpool + base + k_src, kdst + pg * kPageBytes + sub * 1024);
            dma16(vpool + base + v_src, vdst + pg * kPageBytes + sub * 1024);
        } else if (ok) {
            const int64_t base = (int64_t)blk * block_stride + head_off;
            const unsigned char* ks = kpool + base + k_src;
            if (lp * kPage + kPage > P) {           // the page holds new keys
                const int pos = lp * kPage + k_row;  // this lane's key
                if (pos >= P && pos < L) ks = k_new_h + (int64_t)(pos - P) * new_stride + k_chunk;
            }
            dma16(ks, kdst + pg * kPageBytes + sub * 1024);
            if (lp * kPage < P) dma16(vpool + base + v_src, vdst + pg * kPageBytes + sub * 1024);
        }
    };
    auto page_ids = [&](const int ids, int (&blk)[NI]) {
#pragma unroll
        for (int e = 0; e < NI; ++e) blk[e] = __builtin_amdgcn_readlane(ids, page_of(e));
    };
    auto issue_tile = [&](unsigned char* kdst, unsigned char* vdst, int kt, const int ids) {
        int blk[NI];
        page_ids(ids, blk);
#pragma unroll
        for (int e = 0; e < NI; ++e) issue_page(kdst, vdst, kt, blk[e], e);
    };
    // After this wave's loads of tile kt landed: value slots at or past the sequence
    // end become 0 (masked keys get weight 0, and 0 * NaN would poison the product).
    auto zero_tail = [&](unsigned char* vdst, int kt) {
        const int first_bad = L - kt * kBlockN;  // tile-relative key index
        if (first_bad >= kBlockN) return;
#pragma unroll
        for (int e = 0; e < NI; ++e) {
            const int pg = page_of(e);
            const int key0 = pg * kPage + v_half * 8;
            uint16_t* dst = reinterpret_cast<uint16_t*>(vdst + pg * kPageBytes + sub * 1024 + lane * 16);
#pragma unroll
            for (int x = 0; x < 8; ++x)
                if (key0 + x >= first_bad) dst[x] = 0;
        }
    };

    // Fused append, values of new keys. Their rows are token-major, the LDS tile is
    // transposed, so they go through registers: the lanes of a wavefront cover exactly
    // the 1 KiB pieces its own copies fill (32 value rows x 16 keys of one page), one
    // (8 keys, 2 value rows) task per lane and pass: eight 4-byte loads issued with the
    // tile's copies and held during the previous tile's products, then two 16-byte
    // LDS writes (element writes in the group that holds the first new key, whose
    // prefix keys come from the pool). The loads go through a buffer resource over the
    // request's rows, so a key before the prefix end (negative offset) or at or past
    // the sequence end reads as 0 without a test; a tile's offsets stay within
    // (-64, n) rows of the first new key.
    constexpr int kNewTasks = 32 * NI;  // per wavefront and tile
    constexpr int NV = FUSE ? (kNewTasks + 63) / 64 : 1;
    uint32_t nv[NV][8];
    auto has_new = [&](int kt) { return kt * kBlockN + kBlockN > P; };
    auto task_of = [&](int j, int& pg, int& d0, int& half) {
        const int t = lane + 64 * j;
        pg = page_of(t >> 5);
        d0 = 32 * sub + 2 * (t & 15);
        half = (t >> 4) & 1;
        return t < kNewTasks;
    };
    auto load_newv = [&](int kt) {
#pragma unroll
        for (int j = 0; j < NV; ++j) {
            int pg, d0, half;
            const bool ok = task_of(j, pg, d0, half);
            const int key0 = kt * kBlockN + pg * kPage + half * 8;
            const int stride = (int)new_stride;
            const int off = ok ? (key0 - P) * stride + d0 * 2 : INT32_MIN / 2;  // lanes without a task read 0
#pragma unroll
            for (int x = 0; x < 8; ++x) nv[j][x] = __builtin_amdgcn_raw_buffer_load_b32(v_new_r, off + x * stride, 0, 0);
        }
    };
    auto store_newv = [&](unsigned char* vdst, int kt) {
#pragma unroll
        for (int j = 0; j < NV; ++j) {
            int pg, d0, half;
            if (!task_of(j, pg, d0, half)) continue;
            const int key0 = kt * kBlockN + pg * kPage + half * 8;
            if (key0 + 8 <= P) continue;  // eight prefix keys: the page copy holds them
            u32x4 r0, r1;                 // rows d0 and d0 + 1 of the eight keys
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                r0[i] = (nv[j][2 * i] & 0xFFFFu) | (nv[j][2 * i + 1] << 16);
                r1[i] = (nv[j][2 * i] >> 16) | (nv[j][2 * i + 1] & 0xFFFF0000u);
            }
            // d0 is even, so rows d0 and d0 + 1 share the half swap
            unsigned char* row = vdst + pg * kPageBytes + d0 * 32 + ((half ^ ((d0 >> 3) & 1)) * 16);
            if (key0 >= P) {
                *reinterpret_cast<u32x4*>(row) = r0;
                *reinterpret_cast<u32x4*>(row + 32) = r1;
            } else {
                uint16_t* w0 = reinterpret_cast<uint16_t*>(row);
                uint16_t* w1 = reinterpret_cast<uint16_t*>(row + 32);
#pragma unroll
                for (int x = 0; x < 8; ++x)
                    if (key0 + x >= P) {
                        w0[x] = (uint16_t)(nv[j][x] & 0xFFFFu);
                        w1[x] = (uint16_t)(nv[j][x] >> 16);
                    }
            }
        }
    };

    f32x16 o[DB];
    float m_run;   // exponent offset (score * scale * log2(e) units)
    float l_run;   // this lane's half of the row sum of the bf16 weights,
    float l_run1;  // accumulated in two independent sums
    // Exponent offset: a row takes the maximum of its first tile with a visible key and
    // keeps it; the weights of later tiles are exp2 of up to ~100 and fp32 holds their
    // products and sums. If some row's sum leaves that range (a score jump of more than
    // ~100 in log2 units), the work item is run again with the exact running maximum of
    // every tile (rescaled lazily, when it grows by more than 2^8). The final
    // normalisation uses the same offset, so the result does not depend on it.
    bool exact = false;
    const float c = a.scale_log2;
    // key row fed to the QK^T product by this lane: bits 2 and 3 of lr swapped
    const int prow = (lr & 0x13) | ((lr & 4) << 1) | ((lr & 8) >> 1);
    const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};

    // LDS fragment reads kept in flight ahead of their MFMA (fewer when 8-bit codes
    // for the next tile occupy registers during the products; five for bf16 pools at
    // d = 128, measured 0.6-2 % faster than six on the long-prefix workloads)
    constexpr int kAhead = (!FP8 && !FUSE && D == 128) ? 5 : ((FP8 || FUSE) && WAVES == 4 && D == 128) ? 4 : 6;
    // (value fragments: four on the 8-wavefront bf16 tiles at d = 128, where the weights
    // computed between the PV products keep the wavefront busy meanwhile)
    constexpr int kAheadV = (!FP8 && !FUSE && D == 128 && WAVES == 8) ? 4 : kAhead;
    // hook(i) runs after the i-th QK^T product is issued (the next tile's copies go there)
    auto compute_tile = [&](const unsigned char* kb, const unsigned char* vb, int kt, auto&& hook) {
        // S^T = K_tile . Q^T: MFMA i uses K fragment (k = i/2, block b = i%2). Every
        // group below is fenced so the fragment reads stay kAhead MFMAs ahead.
        bf16x8 kf[2 * DK];
        auto kread = [&](int i) {
            const int k = i >> 1, b = i & 1;
            const int krow = 32 * b + prow;
            kf[i] = *reinterpret_cast<const bf16x8*>(kb + krow * (2 * D) + swz_k<D>(2 * k + hh, krow) * 16);
        };
        f32x16 s[2] = {f32x16{}, f32x16{}};
#pragma unroll
        for (int i = 0; i < kAhead; ++i) kread(i);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int i = 0; i < 2 * DK; ++i) {
            if (i + kAhead < 2 * DK) kread(i + kAhead);
            s[i & 1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[i], qf[i >> 1], s[i & 1], 0, 0, 0);
            hook(i);
            __builtin_amdgcn_sched_barrier(0);
        }
        // V fragments of the first value page go out now; they land during the softmax
        bf16x8 vf[4 * DB];
        auto vread = [&](int i) {
            const int st = i / DB, db = i % DB;
            const int d = 32 * db + lr;
            vf[i] = *reinterpret_cast<const bf16x8*>(vb + st * kPageBytes + d * 32 + ((hh ^ ((d >> 3) & 1)) * 16));
        };
#pragma unroll
        for (int i = 0; i < kAheadV; ++i) vread(i);
        __builtin_amdgcn_sched_barrier(0);

        // s[b][e] is the score of tile key 32b + 16(e>>3) + 8hh + (e&7)
        const int key0 = kt * kBlockN;
        if (key0 + kBlockN - 1 > P + it.q0) {
            const int rel = lim - key0 - 8 * hh;
#pragma unroll
            for (int b = 0; b < 2; ++b)
#pragma unroll
                for (int e = 0; e < 16; ++e)
                    s[b][e] = (32 * b + 16 * (e >> 3) + (e & 7) > rel) ? -INFINITY : s[b][e];
        }
        // row maximum: NaN-propagating maxima need no operand canonicalisation and
        // fold three operands per instruction
        if (exact || __any(m_run == -INFINITY)) {
        float mx = s[0][0], mx1 = s[1][0];  // two independent chains
#pragma unroll
        for (int e = 1; e < 16; ++e) {
            mx = __builtin_elementwise_maximum(mx, s[0][e]);
            mx1 = __builtin_elementwise_maximum(mx1, s[1][e]);
        }
        mx = __builtin_elementwise_maximum(mx, mx1);
        {
            const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx), false, false);
            mx = __builtin_elementwise_maximum(__uint_as_float(sw[0]), __uint_as_float(sw[1]));
        }
        const float m_tile = mx * c;
        if (__any(m_tile > m_run + kTileLog2Thresh)) {
            const float m_new = fmaxf(m_run, m_tile);
            // rows that have seen no visible key yet (all -inf; possible in a key chunk
            // that starts past them) hold o = l = 0: any finite alpha keeps them so
            const float alpha = m_new == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m_run - m_new);
            m_run = m_new;
            l_run *= alpha;
            l_run1 *= alpha;
#pragma unroll
            for (int db = 0; db < DB; ++db) o[db] *= alpha;
        }
        }
        const float m_use = (m_run == -INFINITY) ? 0.f : m_run;
        __builtin_amdgcn_sched_barrier(0);

        // O^T += V^T . P^T, one 16-key step st at a time: the weights of step st are
        // computed, then its DB MFMAs are issued with the next step's weights computed
        // between them, in kParts parts (one after every DB / kParts products), so that
        // the exponentials of one step overlap the products of the step before. Quarters
        // for the 8-wavefront bf16 tiles at d = 128, halves otherwise (measured: quarters
        // 1 % faster than halves on the wide tiles, 1.5 % slower on the 128-row ones).
        bf16x8 pf[4];
        constexpr int kParts = (!FP8 && WAVES == 8 && DB >= 4) ? 4 : 2;
        static_assert(DB % kParts == 0 && 4 % kParts == 0, "weight parts");
        // part `part` of step st's eight weights, as bf16, and their row sums: pair q of the
        // step (weights 2q, 2q + 1) goes to l_run for even q and to l_run1 for odd q, in pair
        // order, so the sums do not depend on kParts
        auto weights_part = [&](int st, int part) {
            const int b = st >> 1, e0 = (st & 1) * 8;
#pragma unroll
            for (int e = 8 * part / kParts; e < 8 * (part + 1) / kParts; ++e)
                pf[st][e] = (__bf16)__builtin_amdgcn_exp2f(fmaf(s[b][e0 + e], c, -m_use));
#pragma unroll
            for (int q = 4 * part / kParts; q < 4 * (part + 1) / kParts; ++q) {
                const bf16x2 pq = {pf[st][2 * q], pf[st][2 * q + 1]};
                if (q % 2 == 0) l_run = __builtin_amdgcn_fdot2_f32_bf16(pq, ones, l_run, false);
                else l_run1 = __builtin_amdgcn_fdot2_f32_bf16(pq, ones, l_run1, false);
            }
            // keep the sums here, beside the products (not sunk to the end of the tile)
            asm volatile("" : "+v"(l_run), "+v"(l_run1));
        };
#pragma unroll
        for (int part = 0; part < kParts; ++part) weights_part(0, part);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int st = 0; st < 4; ++st) {
#pragma unroll
            for (int db = 0; db < DB; ++db) {
                const int i = st * DB + db;
                if (i + kAheadV < 4 * DB) vread(i + kAheadV);
                o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[i], pf[st], o[db], 0, 0, 0);
                __builtin_amdgcn_sched_barrier(0);
                if (st + 1 < 4 && (db + 1) % (DB / kParts) == 0) {
                    weights_part(st + 1, (db + 1) / (DB / kParts) - 1);
                    __builtin_amdgcn_sched_barrier(0);
                }
            }
        }
    };

    // 8-bit pools: 16-byte chunks of codes. Chunk c of the K tile is key row
    // c / (D/16), codes 16 (c % (D/16)) ..; chunk c of the V tile is value row c % D
    // of page c / D (16 keys). Lane chunk e is c = 64 (WAVES e + wave) + lane, so a
    // wave's chunks of one e lie in one page.
    constexpr int kChunks = 4 * D;                                   // per tensor and tile
    constexpr int NC = (kChunks + WAVES * 64 - 1) / (WAVES * 64);   // per lane
    const int64_t page_codes = (int64_t)kPage * D;                   // bytes of an 8-bit page
    const int64_t block_codes = (int64_t)a.num_kv_heads * page_codes;
    u32x4 kc8[NC], vc8[NC];
    auto load8 = [&](int kt, const int ids) {
#pragma unroll
        for (int e = 0; e < NC; ++e) {
            const int c0 = 64 * (WAVES * e + wave);  // the wave's first chunk
            const int c = c0 + lane;
            if (c0 < kChunks) {
                const int kpg = (c0 / (D / 16)) / kPage;
                const int vpg = c0 / D;
                int kb = __builtin_amdgcn_readlane(ids, kpg), vb = __builtin_amdgcn_readlane(ids, vpg);
                // pages past the table, past the sequence or with a bad id read block 0
                // (their keys are masked and their values zeroed below)
                const bool kok = kt * 4 + kpg < a.max_blocks && (kt * 4 + kpg) * kPage < L &&
                                 kb >= 0 && kb < a.num_blocks;
                const bool vok = kt * 4 + vpg < a.max_blocks && (kt * 4 + vpg) * kPage < L &&
                                 vb >= 0 && vb < a.num_blocks;
                kb = kok ? kb : 0;
                vb = vok ? vb : 0;
                const uint8_t* kp = reinterpret_cast<const uint8_t*>(a.k_pool) + kb * block_codes +
                                    kvh * page_codes + (c / (D / 16)) % kPage * D + (c % (D / 16)) * 16;
                const uint8_t* vp = reinterpret_cast<const uint8_t*>(a.v_pool) + vb * block_codes +
                                    kvh * page_codes + (c % D) * kPage;
                kc8[e] = *reinterpret_cast<const u32x4*>(kp);
                vc8[e] = *reinterpret_cast<const u32x4*>(vp);
            }
        }
    };
    auto store8 = [&](unsigned char* kdst, unsigned char* vdst, int kt) {
        const int first_bad = L - kt * kBlockN;  // tile-relative key index
#pragma unroll
        for (int e = 0; e < NC; ++e) {
            const int c = 64 * (WAVES * e + wave) + lane;
            if (c < kChunks) {
                u32x4 lo, hi;
                widen_e4m3x16(kc8[e], lo, hi);
                const int kr = c / (D / 16), c8 = c % (D / 16);
                *reinterpret_cast<u32x4*>(kdst + kr * (2 * D) + swz_k<D>(2 * c8, kr) * 16) = lo;
                *reinterpret_cast<u32x4*>(kdst + kr * (2 * D) + swz_k<D>(2 * c8 + 1, kr) * 16) = hi;
                widen_e4m3x16(vc8[e], lo, hi);
                const int pg = c / D, d = c % D;
                const int key0 = pg * kPage;
                if (key0 + kPage > first_bad) {
#pragma unroll
                    for (int x = 0; x < 8; ++x) {
                        const uint32_t keep = (key0 + x < first_bad ? 0xFFFFu : 0u);
                        const uint32_t keep8 = (key0 + 8 + x < first_bad ? 0xFFFFu : 0u);
                        if (x % 2 == 0) {
                            lo[x / 2] &= keep | 0xFFFF0000u;
                            hi[x / 2] &= keep8 | 0xFFFF0000u;
                        } else {
                            lo[x / 2] &= (keep << 16) | 0xFFFFu;
                            hi[x / 2] &= (keep8 << 16) | 0xFFFFu;
                        }
                    }
                }
                unsigned char* vrow = vdst + pg * kPageBytes + d * 32;
                const int sw = (d >> 3) & 1;
                *reinterpret_cast<u32x4*>(vrow + sw * 16) = lo;
                *reinterpret_cast<u32x4*>(vrow + (sw ^ 1) * 16) = hi;
            }
        }
    };

    // Fused append, pool writes: the keys and values of this work item's own tokens
    // (positions P + q0 .. P + q0 + ntok - 1) go from the LDS tile that holds them to
    // their pool slots, bit for bit. Each (token, KV head) has exactly one writer: the
    // query tile that owns the token, in the key chunk that covers its position. bl
    // holds the raw block-table entries of tile kt's four pages (wave-uniform); pages
    // past the table or with a bad id are skipped, as the plain append does.
    auto write_own = [&](const unsigned char* kb, const unsigned char* vb, int kt, const int (&bl)[4]) {
        const int lo = max(P + it.q0, kt * kBlockN), hi = min(P + it.q0 + ntok, kt * kBlockN + kBlockN);
        if (lo >= hi) return;
        constexpr int CPR = D / 8;  // 16-byte chunks per key row
        constexpr int THREADS = WAVES * 64;
        const int64_t page_elems = (int64_t)kPage * D;  // elements of one (block, KV head) page
        int blk4[4];
#pragma unroll
        for (int p = 0; p < 4; ++p)
            blk4[p] = (kt * 4 + p < a.max_blocks && bl[p] >= 0 && bl[p] < a.num_blocks) ? bl[p] : -1;
        auto page_block = [&](int key) {
            const int p = key / kPage - kt * 4;
            return p == 0 ? blk4[0] : p == 1 ? blk4[1] : p == 2 ? blk4[2] : blk4[3];
        };
        for (int u = tid; u < (hi - lo) * CPR; u += THREADS) {
            const int key = lo + u / CPR, c = u % CPR;
            const int b = page_block(key);
            if (b < 0) continue;
            const int rt = key - kt * kBlockN;  // row in the tile
            const u32x4 v = *reinterpret_cast<const u32x4*>(kb + rt * (2 * D) + swz_k<D>(c, rt) * 16);
            *reinterpret_cast<u32x4*>(a.k_dst + ((int64_t)b * a.num_kv_heads + kvh) * page_elems +
                                      (key % kPage) * D + c * 8) = v;
        }
        // values: (page, row d, half h) units of 8 slots
        const int p0 = lo / kPage, np = (hi - 1) / kPage - p0 + 1;
        for (int u = tid; u < np * 2 * D; u += THREADS) {
            const int lp = p0 + u / (2 * D), d = (u % (2 * D)) >> 1, h = u & 1;
            const int k0 = lp * kPage + 8 * h;
            const int a0 = max(k0, lo), a1 = min(k0 + 8, hi);
            if (a0 >= a1) continue;
            const int b = page_block(k0);
            if (b < 0) continue;
            const unsigned char* src = vb + (lp - kt * 4) * kPageBytes + d * 32 + ((h ^ ((d >> 3) & 1)) * 16);
            uint16_t* dst = a.v_dst + ((int64_t)b * a.num_kv_heads + kvh) * page_elems + d * kPage + 8 * h;
            if (a1 - a0 == 8) {
                *reinterpret_cast<u32x4*>(dst) = *reinterpret_cast<const u32x4*>(src);
            } else {
                const uint16_t* s16 = reinterpret_cast<const uint16_t*>(src);
                for (int x = 0; x < 8; ++x)
                    if (k0 + x >= a0 && k0 + x < a1) dst[x] = s16[x];
            }
        }
    };

    // One pipeline step: start the next tile's loads into the other buffers, compute
    // this tile, make the next tile visible.
    // (ids: block-table entries of the next tile to copy, entry p in lanes with lane % 4 == p)
    int bl_cur[4];  // (fused append) the entries of the tile being computed, wave-uniform
    auto take_ids = [&](int (&bl)[4]) {
#pragma unroll
        for (int p = 0; p < 4; ++p) bl[p] = __builtin_amdgcn_readlane(ids, p);
    };
    int kt = it.kt_begin;
    auto step = [&](unsigned char* kc, unsigned char* vc, unsigned char* kn, unsigned char* vn) {
        const bool more = kt + 1 < it.kt_end;
        int bl_next[4];
        if constexpr (FUSE) take_ids(bl_next);
        // the next tile's block ids, read before any copy of this step is in flight (the
        // compiler waits for every outstanding load before reading `ids`)
        int nb[NI];
        page_ids(ids, nb);
        if (more) {
            if constexpr (FP8) {
                load8(kt + 1, ids);
                if (kt + 2 < it.kt_end) fetch_ids(kt + 2, ids);
            }
            if constexpr (FUSE)
                if (has_new(kt + 1)) load_newv(kt + 1);
        }
        if constexpr (FUSE) write_own(kc, vc, kt, bl_cur);
        // bf16 pools: the next tile's copies are issued between the first products of
        // this one (piece e after product 3e + 2; 3e + 1 with the append fused in), then
        // the table entries of the tile after
        static_assert(3 * NI < 2 * DK, "copies fit between the QK^T products");
        constexpr int kCopyAt = FUSE ? 1 : 2;
        compute_tile(kc, vc, kt, [&](int i) {
            if constexpr (!FP8) {
                if (i % 3 == kCopyAt && i / 3 < NI) {
                    if (more) issue_page(kn, vn, kt + 1, nb[i / 3], i / 3);
                } else if (i == 3 * NI) {
                    if (kt + 2 < it.kt_end) fetch_ids(kt + 2, ids);
                }
            }
        });
        if (more) {
            if constexpr (FP8) {
                store8(kn, vn, kt + 1);
            } else {
                wait_vmem<0>();
                if constexpr (FUSE)
                    if (has_new(kt + 1)) store_newv(vn, kt + 1);
                zero_tail(vn, kt + 1);
            }
        }
        __syncthreads();
        if constexpr (FUSE)
#pragma unroll
            for (int p = 0; p < 4; ++p) bl_cur[p] = bl_next[p];
    };

    for (;;) {
#pragma unroll
    for (int db = 0; db < DB; ++db) o[db] = f32x16{};
    m_run = -INFINITY;
    l_run = 0.f;
    l_run1 = 0.f;
    kt = it.kt_begin;
    if (exact) fetch_ids(kt, ids);  // the first pass has them from the start
    if constexpr (FP8) {
        load8(kt, ids);
        if (kt + 1 < it.kt_end) fetch_ids(kt + 1, ids);
        store8(k_lds0, v_lds0, kt);
    } else {
        issue_tile(k_lds0, v_lds0, kt, ids);
        if constexpr (FUSE) take_ids(bl_cur);
        if constexpr (FUSE)
            if (has_new(kt)) load_newv(kt);
        if (kt + 1 < it.kt_end) fetch_ids(kt + 1, ids);
        wait_vmem<0>();
        if constexpr (FUSE)
            if (has_new(kt)) store_newv(v_lds0, kt);
        zero_tail(v_lds0, kt);
    }
    __syncthreads();
    while (true) {
        step(k_lds0, v_lds0, k_lds1, v_lds1);
        if (++kt >= it.kt_end) break;
        step(k_lds1, v_lds1, k_lds0, v_lds0);
        if (++kt >= it.kt_end) break;
    }
    if (exact || !__syncthreads_or(!(l_run + l_run1 <= 0x1p100f))) break;
    exact = true;
    }

    l_run += l_run1;
    const float l_tot = l_run + __shfl_xor(l_run, 32);
    const float inv = l_tot > 0.f ? a.v_scale / l_tot : 0.f;  // v_scale is 1 for bf16 pools
    const float lse_v = l_tot > 0.f ? (m_run + log2f(l_tot)) * kLn2 : -INFINITY;
    // o[db][4j + i] is element d = 32db + 8j + 4hh + i of this lane's row
    if (it.part < 0) {
        // Output rows go through LDS so that every store writes whole rows: a lane's own
        // values cover 16 bytes of each of 32 rows, 256 bytes apart. The tiles are no
        // longer read (the last barrier above), so each wavefront takes 8 KiB (4 KiB for
        // d = 64) of the tile buffers: its 32 rows, 16-byte chunks XOR-swizzled by row.
        // Each store then covers 256 (128) contiguous bytes of 4 (8) rows, and the rows
        // of one token's query heads are adjacent in the output.
        constexpr int RB = 2 * D;                       // bytes per row
        constexpr int CH = RB / 16;                     // 16-byte chunks per row
        constexpr int kStage = kRowsPerWave * RB;       // bytes per wavefront
        constexpr int kPerBuf = kTileBytes / kStage;    // wavefronts per tile buffer
        static_assert(kPerBuf * 4 >= WAVES && kPerBuf * kStage == kTileBytes, "stage layout");
        const int sb = wave / kPerBuf;
        unsigned char* stage = (sb == 0 ? k_lds0 : sb == 1 ? v_lds0 : sb == 2 ? k_lds1 : v_lds1) +
                               (wave % kPerBuf) * kStage;
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                u32x2 w;
                w[0] = pack_bf16x2(o[db][4 * j] * inv, o[db][4 * j + 1] * inv);
                w[1] = pack_bf16x2(o[db][4 * j + 2] * inv, o[db][4 * j + 3] * inv);
                *reinterpret_cast<u32x2*>(stage + lr * RB + ((4 * db + j) ^ (lr & (CH - 1))) * 16 + 8 * hh) = w;
            }
        if (row_ok && a.lse != nullptr && hh == 0) a.lse[qrow] = lse_v;
        wave_lds_sync();
        constexpr int kRowsPerStore = 64 / CH;
#pragma unroll
        for (int i = 0; i < kRowsPerWave / kRowsPerStore; ++i) {
            const int rr = i * kRowsPerStore + lane / CH, ch = lane % CH;
            const u32x4 v = *reinterpret_cast<const u32x4*>(stage + rr * RB + (ch ^ (rr & (CH - 1))) * 16);
            const int mr = wave * kRowsPerWave + rr;  // the stored row's token and head
            const int tr = mr / a.group;
            if (tr < ntok) {
                const int64_t qr = (int64_t)(cu + it.q0 + tr) * a.num_q_heads + kvh * a.group + (mr - tr * a.group);
                *reinterpret_cast<u32x4*>(a.out + qr * D + ch * 8) = v;
            }
        }
    } else {
        // Partial rows (fp32) of a split item, through the same stage: the wavefront's 32
        // rows are contiguous in the partial buffer, so each store covers whole rows; rows
        // larger than the stage go in rounds of kRows.
        constexpr int RB = 4 * D;                             // bytes per fp32 row
        constexpr int CH = RB / 16;                           // 16-byte chunks per row
        constexpr int kStage = 4 * kTileBytes / WAVES;        // stage bytes per wavefront
        constexpr int kRows = kStage / RB < kRowsPerWave ? kStage / RB : kRowsPerWave;
        static_assert(kRows >= 2 && kRowsPerWave % kRows == 0 && (kRows * CH) % 64 == 0, "partial stage");
        constexpr int kPerBuf = kTileBytes / kStage;
        const int sb = wave / kPerBuf;
        unsigned char* stage = (sb == 0 ? k_lds0 : sb == 1 ? v_lds0 : sb == 2 ? k_lds1 : v_lds1) +
                               (wave % kPerBuf) * kStage;
        const int64_t prow0 = ((int64_t)it.part * a.num_kv_heads + kvh) * kBlockRows + wave * kRowsPerWave;
        constexpr int kSw = CH < 16 ? CH : 16;                // chunk swizzle span
#pragma unroll
        for (int r0 = 0; r0 < kRowsPerWave; r0 += kRows) {
            if (lr >= r0 && lr < r0 + kRows) {
                const int sr = lr - r0;
#pragma unroll
                for (int db = 0; db < DB; ++db)
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        f32x4 w = {o[db][4 * j] * inv, o[db][4 * j + 1] * inv, o[db][4 * j + 2] * inv,
                                   o[db][4 * j + 3] * inv};
                        const int ch = (8 * db + 2 * j + hh) ^ (sr & (kSw - 1));
                        *reinterpret_cast<f32x4*>(stage + sr * RB + ch * 16) = w;
                    }
            }
            wave_lds_sync();
#pragma unroll
            for (int i = 0; i < kRows * CH / 64; ++i) {
                const int c = i * 64 + lane, sr = c / CH, ch = c % CH;
                const f32x4 v = *reinterpret_cast<const f32x4*>(stage + sr * RB + (ch ^ (sr & (kSw - 1))) * 16);
                *reinterpret_cast<f32x4*>(a.part_o + (prow0 + r0 + sr) * D + ch * 4) = v;
            }
            wave_lds_sync();  // the next round overwrites the stage
        }
        if (hh == 0) a.part_lse[prow0 + lr] = lse_v;
    }
}

template <int D, int WAVES, bool FP8>
__global__ __launch_bounds__(WAVES * 64, 8 / WAVES) void attention_kernel(const AttnArgs a) {
    attention_body<D, WAVES, FP8, false>(a, blockIdx.x);
}

// Attention with the KV append fused in: the work items read new keys from the new
// tokens' arrays (so they do not wait for any append) and write their own tokens'
// keys and values into the pools from LDS.
template <int D, int WAVES>
__global__ __launch_bounds__(WAVES * 64, 8 / WAVES) void attention_append_kernel(const AttnArgs a) {
    attention_body<D, WAVES, false, true>(a, blockIdx.x);
}

// Merge the key chunks of one split query tile: with m = max_s lse_s,
// lse = m + log sum_s exp(lse_s - m) and o = sum_s exp(lse_s - m) o_s / sum_s exp(lse_s - m),
// in a fixed chunk order (deterministic).

// Resident launch (wide tiles): one workgroup per compute unit, each
// taking work items until none is left. Queue x holds the regular launch's indices
// x, x + 8, x + 16, ...: the hardware deals workgroups to the eight XCDs in turn, so
// workgroup b serves queue b % 8 and each XCD runs the items (and KV heads) it runs in
// the regular launch, keeping their K/V in its L2. A workgroup whose queue is empty
// takes items from the other queues, so XCDs that run slower do not hold up the end of
// the launch; and a freed compute unit starts its next item without waiting for the
// dispatcher, which hands out new workgroups in index order across the XCDs. Tickets
// are agent-scope atomics on the workspace's counters; the last workgroup to leave
// sets them back to zero for the next launch (the ticket atomics of every other
// workgroup returned before it counted itself out).
template <int D, bool FP8>
__global__ __launch_bounds__(kWideWaves * 64, 1) void attention_resident_kernel(const AttnArgs a, int total) {
    __shared__ int s_tk, s_empty;
    const int x = (int)(blockIdx.x % (unsigned)kQueues);
    if (threadIdx.x == 0) s_empty = 0;
    for (;;) {
        if (threadIdx.x == 0) {
            int b = -1, empty = s_empty;
            for (int j = 0; j < kQueues && b < 0; ++j) {
                const int y = (x + j) % kQueues;
                if (empty & (1 << y)) continue;
                const int k = __hip_atomic_fetch_add(&a.queues[y], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                if ((int64_t)k * kQueues + y < total) b = k * kQueues + y;
                else empty |= 1 << y;
            }
            s_empty = empty;
            s_tk = b;
        }
        __syncthreads();
        const int b = s_tk;
        __syncthreads();  // every wavefront has read the ticket before the next one is written
        if (b < 0) break;
        attention_body<D, kWideWaves, FP8, false>(a, (unsigned)b);
    }
    if (threadIdx.x == 0) {
        const int out = __hip_atomic_fetch_add(&a.queues[kQueues], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (out == (int)gridDim.x - 1)
            for (int y = 0; y <= kQueues; ++y)
                __hip_atomic_store(&a.queues[y], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}

// A workgroup merges kCombineRows rows of one (query tile, KV head); a thread
// owns four consecutive output elements of one row, so the partial rows are
// read with coalesced 16-byte loads.
template <int D>
__global__ __launch_bounds__(kCombineThreads) void combine_kernel(const CombineArgs a) {
    constexpr int CPR = D / 4;                      // float4 chunks per row
    constexpr int kRows = kCombineThreads / CPR;    // rows per workgroup
    const int groups = ceil_div(a.block_m, kRows);
    const unsigned tile = blockIdx.x / (unsigned)groups;
    const int m = (int)(blockIdx.x % (unsigned)groups) * kRows + (int)threadIdx.x / CPR;
    if (m >= a.block_m) return;
    const int c4 = (int)threadIdx.x % CPR;
    const int kvh = (int)(tile % (unsigned)a.num_kv_heads);
    const CombineItem ci = a.combines[tile / (unsigned)a.num_kv_heads];
    if (ci.ns <= 0 || ci.r < 0 || ci.r >= a.batch || ci.q0 < 0 || ci.part_base < 0 ||
        ci.part_base + ci.ns > a.num_partials)
        return;
    const int cu = a.cu_new_lens[ci.r];
    const int n = a.cu_new_lens[ci.r + 1] - cu;
    if (ci.q0 >= n) return;
    const int ntok = min(a.tq, n - ci.q0);
    const int t = m / a.group, hl = m - t * a.group;
    if (t >= ntok) return;
    const int64_t row0 = ((int64_t)ci.part_base * a.num_kv_heads + kvh) * a.block_m + m;
    const int64_t split_stride = (int64_t)a.num_kv_heads * a.block_m;  // rows between chunks
    // chunks are read kBatch at a time with independent loads (the merge is bound by
    // memory latency, not arithmetic); the sums still run in chunk order
    constexpr int kBatch = 8;
    float mx = -INFINITY;
    for (int s0 = 0; s0 < ci.ns; s0 += kBatch) {
        float l[kBatch];
#pragma unroll
        for (int u = 0; u < kBatch; ++u)
            l[u] = s0 + u < ci.ns ? a.part_lse[row0 + (s0 + u) * split_stride] : -INFINITY;
#pragma unroll
        for (int u = 0; u < kBatch; ++u) mx = fmaxf(mx, l[u]);
    }
    float tot = 0.f;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int s0 = 0; s0 < ci.ns; s0 += kBatch) {
        float l[kBatch];
        f32x4 v[kBatch];
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            const bool ok = s0 + u < ci.ns;
            const int64_t pr = row0 + (int64_t)(ok ? s0 + u : s0) * split_stride;
            l[u] = ok ? a.part_lse[pr] : -INFINITY;
            v[u] = *reinterpret_cast<const f32x4*>(a.part_o + pr * D + 4 * c4);
        }
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            const float w = expf(l[u] - mx);  // 0 for the padding entries
            tot += w;
            acc += w * v[u];
        }
    }
    const float lse_tot = mx + logf(tot);
    acc *= 1.f / tot;
    const int64_t qrow = (int64_t)(cu + ci.q0 + t) * a.num_q_heads + kvh * a.group + hl;
    u32x2 w2;
    w2[0] = pack_bf16x2(acc[0], acc[1]);
    w2[1] = pack_bf16x2(acc[2], acc[3]);
    *reinterpret_cast<u32x2*>(a.out + qrow * D + 4 * c4) = w2;
    if (a.lse != nullptr && c4 == 0) a.lse[qrow] = lse_tot;
}

}  // namespace
}  // namespace gc
