// Device body of the causal prefill attention (one work-group of it), shared
// by the prefill kernel and the fused prefill + decode kernel.
//
// Prefill is compute-bound (paper Sec. 2.2; Sec. 3.3, Table
// "tab:theory_cost": O(n d^2 + L n d) with L = r + n), so both contractions
// run on the bf16 matrix cores (fp32 accumulate).
//
// Work-group = 8 waves; a query block = 64 query positions x 4 query heads of
// one kv head; wave w owns head (w % 4) of the group and positions
// 32*(w / 4) .. +31 of the block, so every K/V tile staged in LDS serves
// 4 heads x 64 positions.  Each work-group processes two blocks of the same
// heads, block nqb-1-i and block i: causal blocks grow linearly with the block
// index, so all pairs cost about the same and the grid has no long tail.
// Each wave's state (Q^T, S, P, O) stays in registers.
//
// Per key tile t (all waves, one work-group barrier per tile):
//     S(t)^T = K(t) Q^T;  mask, online softmax of S(t) -> P(t) (bf16);
//     O^T += V(t)^T P(t)^T
// Key tiles of 64 keys = 4 pages go from HBM straight into LDS with the direct
// buffer-to-LDS loads, double-buffered: the loads of tile t+1 are issued
// between the MFMAs of S(t) and waited for at the end of tile t; the first
// tile of a block is requested before Q and the block-table copy are read.
// Rows are 256 B with their 16-byte chunks permuted by XOR with
// swz(r) = 4(r%4) ^ (r/4)%4, which makes both the 16-byte K operand reads and
// the transposing V reads bank-conflict free; the permutation is applied on
// the HBM side of each load.  The 16 MFMAs of each product issue in a fixed
// order with the LDS operands of the next few already in flight.
//   S^T[key][q] = K Q^T      32x32x16 MFMA; A = K rows from LDS, B = Q^T
//   O^T[d][q] += V^T P^T     32x32x16 MFMA; A = V^T gathered by the LDS
//                            transposing read (ds_read_b64_tr_b16), B = P^T
//                            taken straight from the S^T accumulators as bf16
// Online softmax in base 2 (scores scaled by scale*log2 e inside one FMA); the
// causal mask is applied only on tiles that cross the diagonal; row sums are
// taken over the bf16 probabilities the PV product uses.  The running
// maximum moves only when a column's tile maximum exceeds it by more than 2^8
// (O and l are then rescaled); O / l does not depend on the reference maximum.
// O is staged through LDS so that each store writes whole 256-byte rows.
// Causal position: query row i of a sequence with prefix r sees keys
// 0 .. r + i (bottom-right alignment; a chunk reads every earlier chunk's KV).
#pragma once
#include <type_traits>

#include "mw_internal.h"

namespace {
namespace pf {

using namespace mw;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kWaves = 8;
constexpr int kThreads = 64 * kWaves;
constexpr int BM = 64;                       // query positions per 8-wave work-group
constexpr int BN = 64;                       // keys per tile
constexpr int ROW = kHeadDim;                // tile row = one key, 128 bf16 (256 B)
constexpr int TILE = BN * ROW;               // one K or V tile, bf16 elements
constexpr int kBtCache = 4096;               // block-table entries staged in LDS
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kRescaleLog2 = 8.f;          // lazy-rescale threshold (log2 units)

typedef __attribute__((address_space(3))) void lds_void;
constexpr int kBufferFormat = 0x00020000;    // buffer descriptor word 3: 32-bit data format

constexpr int kAhead = 4;                    // MFMA operands kept in flight

template <bool B>
using flag = std::integral_constant<bool, B>;

// Where a piece of a key-range-split query block leaves its partial result:
// the unnormalised output O~ = sum_j 2^(s_j - m) v_j and (m, l = sum_j
// 2^(s_j - m)) over the piece's keys (s in log2 units), for every row and
// query head, in slot `piece`.
struct SplitOut {
    float *o;     // [max_pieces][rows][hq][128] fp32
    float2 *ml;   // [max_pieces][rows][hq]
    int64_t rows; // rows of the call (sum of the new lengths)
    int piece_tiles, max_pieces, piece;
};

__device__ inline int swz(int row) { return ((row & 3) << 2) ^ ((row >> 2) & 3); }

__device__ inline uint32_t cvt2(float a, float b) {
    bf16x2 v;
    v[0] = static_cast<__bf16>(a);
    v[1] = static_cast<__bf16>(b);
    return __builtin_bit_cast(uint32_t, v);
}

// NaN-propagating maximum: a single v_maximum3_f32 on gfx950, with no
// canonicalisation of the MFMA results it reads.
__device__ inline float vmax(float a, float b) { return __builtin_elementwise_maximum(a, b); }

// max(x, x of lane l ^ 32).  v_permlane32_swap exchanges lanes 32..63 of its
// first operand with lanes 0..31 of its second, so with x in both operands
// one result holds the lower half's values in every lane and the other the
// upper half's.  Inline assembly because this compiler takes the builtin's
// second result to be its first (the maximum would then cover only half the
// keys); the s_nop covers the two wait states the swap needs after a vector
// instruction writes its operands.
__device__ inline float max_xor32(float x) {
    float a = x, b = x;
    asm volatile("s_nop 1\n\tv_permlane32_swap_b32 %0, %1" : "+v"(a), "+v"(b));
    return vmax(a, b);
}

// Transposing LDS read: within each 16-lane group, lane s points at 4
// consecutive elements of a row; lane 4a+b receives element b of the chunks of
// lanes a, a+4, a+8, a+12.  The address-space cast keeps the pointer's origin
// visible to the compiler.
__device__ inline i16x4 lds_read_tr(const char *p) {
    return __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4 *)(p));
}

// Work-group barrier without the memory fence of __syncthreads: LDS reads are
// consumed before every barrier, and the tile loads are waited for explicitly.
__device__ inline void wg_barrier() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// kTableInLds: every block-table entry the work-group needs fits the LDS copy.
// The other instantiation reads entries past it with scalar loads, which makes
// the compiler wait for all outstanding LDS reads wherever it needs one.
// NW: waves per work-group.  8 (query blocks of 64 positions; waves w and
// w+4 share a SIMD) or 4 (blocks of 32 positions, two work-groups per CU):
// the same per-wave work, for grids that would leave CUs idle with 8.
// kSplit (4 waves only): the work-group computes piece sp.piece of its query
// block's key range (prefill_pieces), writing partials to sp when the block
// has more than one piece and the normalised output otherwise.
template <bool kTableInLds, int NW, bool kSplit = false>
__device__ __forceinline__ void
prefill_block(const uint16_t *__restrict__ kpool, const uint16_t *__restrict__ vpool,
              const uint16_t *__restrict__ q, uint16_t *__restrict__ out,
              const int32_t *__restrict__ qo_indptr, const int32_t *__restrict__ prefix_lens,
              const int32_t *__restrict__ bt, int bt_stride, int hkv, int group, int num_pages,
              float scale_log2, int paired, int n_hgroups,
              // work-group coordinates (x: query block and heads, b: sequence)
              // and the LDS buffers: K and V tiles (2 * TILE each, 1024-byte
              // aligned) and the block-table copy (kBtCache entries)
              const int x, const int b, uint16_t *s_k, uint16_t *s_v, int32_t *s_bt, const SplitOut sp = {}) {
    static_assert(NW == 8 || NW == 4, "8 or 4 waves");
    static_assert(!kSplit || NW == 4, "the key-range split runs 4-wave blocks");
    constexpr int kBM = 8 * NW;         // query positions per block
    constexpr int kNT = 64 * NW;        // threads
    constexpr int kRows = 64 / NW;      // tile rows (keys) each wave loads
    constexpr int kJ = kRows / 4;       // 1-KB loads per wave per K (or V) tile
    constexpr int kEvery = 8 / kJ;      // QK MFMAs between two of this wave's loads
    // Work-group = one query block of one (sequence, kv head, head group),
    // heaviest blocks first, or (paired) the pair of blocks nqb-1-i and i:
    // causal blocks grow linearly with the block index, so every pair costs
    // about the same number of key tiles.
    const int kvh = x % hkv;
    const int hg = (x / hkv) % n_hgroups;
    const int pair = x / (hkv * n_hgroups);
    const int row0 = qo_indptr[b];
    const int n = qo_indptr[b + 1] - row0;
    const int nqb = (n + kBM - 1) / kBM;
    if (pair >= (paired ? (nqb + 1) / 2 : nqb)) return;
    const int n_items = (!paired || pair == nqb - 1 - pair) ? 1 : 2;
    const int r = prefix_lens[b];
    // key tiles [t_lo, t_hi) of this work-group's (single) block and its
    // number of pieces (1 without the split); tile t_lo is loaded first and
    // page p of the sequence sits at s_bt[p - 4 t_lo] in the table copy
    int t_lo = 0, t_hi = 0, n_pieces = 1;
    if constexpr (kSplit) {
        const int nt_b = prefill_block_tiles(r, n, nqb - 1 - pair);
        n_pieces = prefill_pieces(nt_b, sp.piece_tiles, sp.max_pieces);
        if (sp.piece >= n_pieces) return;
        t_lo = sp.piece * nt_b / n_pieces;
        t_hi = (sp.piece + 1) * nt_b / n_pieces;
    }
    const int pbase = 4 * t_lo;
    const int32_t *btrow = bt + static_cast<size_t>(b) * bt_stride;
    const int np_seq = min((r + n + kPageSize - 1) / kPageSize, bt_stride);

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // uniform per wave
    const int hl = hg * 4 + (wave & 3);  // head within the kv group
    const bool active = hl < group;
    const int hq = hkv * group;
    const int h = kvh * group + (active ? hl : 0);
    const int l32 = lane & 31, g = lane >> 5;

    // block-table entries of this work-group's keys (the heavier block's)
    {
        const int nt_a = (r + min((nqb - pair) * kBM, n) + BN - 1) / BN;
        const int np_wg = min(4 * (kSplit ? t_hi : nt_a), np_seq);
        for (int i = pbase + threadIdx.x; i < min(np_wg, pbase + kBtCache); i += kNT) s_bt[i - pbase] = btrow[i];
    }
    const int seq_len = r + n;

    // ---- per-lane byte offsets, computed once
    // K operand: row l32 (+32 rows for the second key block), logical chunk
    // 2kb+g; since 2kb+g = 2kb ^ g, dim-step kb is at koff ^ 32kb
    const int koff = l32 * 256 + 16 * (g ^ swz(l32));
    // V transposing reads: lane s of 16-lane group q reads row 8hh + 4(q/2) + s/4
    // (+16 ks) at dims 32db + 16(q%2) + 4(s%4): logical chunk 4db + 2(q%2) + (s%4)/2,
    // so dim block db is at voff[hh] ^ 64db
    int voff[2];
    {
        const int q16 = lane >> 4, s16 = lane & 15;
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
            const int row = 8 * hh + 4 * (q16 >> 1) + (s16 >> 2);
            const int chunk = (2 * (q16 & 1) + ((s16 & 3) >> 1)) ^ swz(row);
            voff[hh] = row * 256 + 16 * chunk + 8 * (s16 & 1);
        }
    }
    // direct loads: wave w moves rows kRows w + 4j + lane/16 (j < kJ) of every
    // K and V tile, all in page kRows w / 16 of the tile; lane i lands in
    // physical chunk i%16.  Byte offsets within the page:
    int goff[kJ];
#pragma unroll
    for (int j = 0; j < kJ; ++j) {
        const int row = (kRows * wave) % 16 + 4 * j + (lane >> 4);
        goff[j] = 2 * (row * kHeadDim + 8 * ((lane & 15) ^ swz(row)));
    }
    const int lpage = kRows * wave / 16;  // page of the tile this wave loads

    // per-item state
    int qblk = 0, nt = 0, pos = 0, qabs = 0, diag = 0;
    uint4 qop[8];
    f32x16 oacc[4];
    f32x16 sacc[2];
    uint4 pop[4];
    float m_run = -INFINITY;
    float l_run = 0.f;

    // The (page, kv head) block of sequence page p (uniform per wave): its pool
    // element offset and the bytes of it that hold the sequence's tokens.  A
    // page past the sequence or outside the pool has 0 bytes, and the last page
    // only its rows below r + n: the buffer loads return zeros past that, so
    // slack slots and absent pages are never read, whatever bits they hold
    // (zero keys and values past the sequence are also discarded by the causal
    // mask: they lie after every query).
    struct PageRef {
        size_t base;
        int bytes;
    };
    auto page_ref = [&](int p, int page) __attribute__((always_inline)) {
        const bool ok = p < np_seq && page >= 0 && page < num_pages;
        PageRef ref;
        ref.base = ok ? (static_cast<size_t>(page) * hkv + kvh) * (kPageSize * kHeadDim) : 0;
        ref.bytes = ok ? min(seq_len - kPageSize * p, kPageSize) * (kHeadDim * 2) : 0;
        return ref;
    };
    // Page `lpage` of key tile `it`, its entry read from the LDS copy of the table.
    auto tile_page = [&](int it) __attribute__((always_inline)) {
        const int p = 4 * it + lpage;
        int page = -1;
        if (p < np_seq) {
            if constexpr (kTableInLds)
                page = __builtin_amdgcn_readfirstlane(s_bt[p - pbase]);
            else
                page = p - pbase < kBtCache ? __builtin_amdgcn_readfirstlane(s_bt[p - pbase]) : btrow[p];
        }
        return page_ref(p, page);
    };
    // Loads (1 KB each) of this wave's half page of one tile: buffer loads over
    // a descriptor of the page's valid rows (the hardware returns zeros past
    // them).  Buffer rather than global loads: the compiler counts a global
    // load into LDS as an outstanding LDS access too, which would make every
    // operand read wait for all LDS reads in flight.  The LDS destination goes
    // through an integer, so the compiler does not tie later LDS reads to these
    // loads; the loop waits for them explicitly.
    auto page_rsrc = [&](const uint16_t *pool, PageRef ref) __attribute__((always_inline)) {
        return __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t *>(pool + ref.base), 0, ref.bytes,
                                                 kBufferFormat);
    };
    auto page_load = [&](__amdgpu_buffer_rsrc_t rsrc, uint16_t *dst, int j) __attribute__((always_inline)) {
        __builtin_amdgcn_raw_ptr_buffer_load_lds(
            rsrc, reinterpret_cast<lds_void *>(reinterpret_cast<uintptr_t>(dst + (kRows * wave + 4 * j) * ROW)), 16,
            goff[j], 0, 0, 0);
    };

    // Matrix work: O^T += V^T P^T with V from tile buffer vbuf (if PV), then
    // S^T = K Q^T with K from tile buffer kbuf (if QK); `load(j)` is called
    // after every kEvery-th MFMA of a QK-only phase.  Operation i < npv is PV
    // key-step i/4, dim block i%4; the rest are QK dim-step j/2, key block j%2.
    auto mfma_phase = [&](auto pv_flag, auto qk_flag, int kbuf, int vbuf, auto load) __attribute__((always_inline)) {
        constexpr bool PV = decltype(pv_flag)::value, QK = decltype(qk_flag)::value;
        constexpr int npv = PV ? 16 : 0;
        constexpr int nop = npv + (QK ? 16 : 0);
        const char *vb_ = reinterpret_cast<const char *>(s_v + vbuf * TILE);
        const char *kb_ = reinterpret_cast<const char *>(s_k + kbuf * TILE);
        // per-read offsets are recomputed here (one XOR each) rather than held
        // in registers across the loop
        int ko = koff, vo0 = voff[0], vo1 = voff[1];
        asm volatile("" : "+v"(ko), "+v"(vo0), "+v"(vo1));
        auto fetch = [&](int i) __attribute__((always_inline)) -> bf16x8 {
            if (i < npv) {
                const int off = (i >> 2) * 16 * 256;
                const i16x4 lo = lds_read_tr(vb_ + off + (vo0 ^ (64 * (i & 3))));
                const i16x4 hi = lds_read_tr(vb_ + off + (vo1 ^ (64 * (i & 3))));
                return __builtin_bit_cast(
                    bf16x8, make_uint4(__builtin_bit_cast(uint2, lo).x, __builtin_bit_cast(uint2, lo).y,
                                       __builtin_bit_cast(uint2, hi).x, __builtin_bit_cast(uint2, hi).y));
            }
            const int j = i - npv;
            return *reinterpret_cast<const bf16x8 *>(kb_ + (j & 1) * 32 * 256 + (ko ^ (32 * (j >> 1))));
        };
        __builtin_amdgcn_s_setprio(2);  // a wave issuing MFMAs wins issue conflicts on the SIMD
        bf16x8 opnd[kAhead];
#pragma unroll
        for (int i = 0; i < kAhead; ++i) opnd[i] = fetch(i);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int i = 0; i < nop; ++i) {
            const bf16x8 a = opnd[i % kAhead];
            if (i < npv) {
                oacc[i & 3] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                    a, __builtin_bit_cast(bf16x8, pop[i >> 2]), oacc[i & 3], 0, 0, 0);
            } else {
                // the first step of each key block starts from zero, so the
                // score registers are free until the QK half of the phase
                const int j = i - npv;
                const f32x16 zero = {};
                sacc[j & 1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                    a, __builtin_bit_cast(bf16x8, qop[j >> 1]), j < 2 ? zero : sacc[j & 1], 0, 0, 0);
            }
            if (i + kAhead < nop) opnd[i % kAhead] = fetch(i + kAhead);
            if (!PV && i % kEvery == kEvery - 1) load(i / kEvery);
            __builtin_amdgcn_sched_barrier(0);
        }
        __builtin_amdgcn_s_setprio(0);
    };

    // Causal mask and online softmax of S(t) into P(t).
    auto softmax_phase = [&](int t) __attribute__((always_inline)) {
        const int k0 = t * BN;
        if (k0 + BN - 1 > diag) {
#pragma unroll
            for (int blk = 0; blk < 2; ++blk)
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const int key = k0 + 32 * blk + 8 * (i >> 2) + 4 * g + (i & 3);
                    if (key > qabs) sacc[blk][i] = -INFINITY;
                }
        }
        // column maximum as a tree of 3-way maxima (short dependency chain)
        float m8[8];
#pragma unroll
        for (int j = 0; j < 8; ++j)
            m8[j] = vmax(vmax(sacc[j >> 2][4 * (j & 3)], sacc[j >> 2][4 * (j & 3) + 1]),
                         vmax(sacc[j >> 2][4 * (j & 3) + 2], sacc[j >> 2][4 * (j & 3) + 3]));
        float mx = vmax(vmax(vmax(m8[0], m8[1]), vmax(m8[2], m8[3])), vmax(vmax(m8[4], m8[5]), vmax(m8[6], m8[7])));
        mx = max_xor32(mx);  // lanes l and l^32 hold the same query
        const float m_tile = mx * scale_log2;
        if (__builtin_amdgcn_ballot_w64(m_tile > m_run + kRescaleLog2) != 0) {
            const float m_new = vmax(m_run, m_tile);
            const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
            m_run = m_new;
            l_run *= alpha;
#pragma unroll
            for (int db = 0; db < 4; ++db)
#pragma unroll
                for (int i = 0; i < 16; ++i) oacc[db][i] *= alpha;
        }
        // key-step ks covers registers 8a..8a+7 of block ks/2, i.e. keys
        // 16ks + 8(e/4) + 4g + e%4 for operand element e
        float lsum[4];
#pragma unroll
        for (int kstep = 0; kstep < 4; ++kstep) {
            const int blk = kstep >> 1, a8 = (kstep & 1) * 8;
            float p[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) p[e] = __builtin_amdgcn_exp2f(fmaf(sacc[blk][a8 + e], scale_log2, -m_run));
            pop[kstep] = make_uint4(cvt2(p[0], p[1]), cvt2(p[2], p[3]), cvt2(p[4], p[5]), cvt2(p[6], p[7]));
            // row sums in fp32 with plain adds: a dot product over the bf16
            // values would wait behind the other wave's MFMAs on this SIMD
            lsum[kstep] = ((p[0] + p[1]) + (p[2] + p[3])) + ((p[4] + p[5]) + (p[6] + p[7]));
        }
        l_run += (lsum[0] + lsum[1]) + (lsum[2] + lsum[3]);
    };

    // The first tile of an item: its pages straight from the block table in
    // HBM, so the loads can start before the table copy in LDS is complete
    // (its K and, with 4 waves, its V; the 8-wave body loads V(0) in its
    // first period).
    auto first_tile = [&](auto with_v) __attribute__((always_inline)) {
        const int p0 = pbase + lpage;
        const PageRef ref = page_ref(p0, p0 < np_seq ? btrow[p0] : -1);
        const __amdgpu_buffer_rsrc_t rk = page_rsrc(kpool, ref), rv = page_rsrc(vpool, ref);
#pragma unroll
        for (int j = 0; j < kJ; ++j) {
            page_load(rk, s_k, j);
            if constexpr (decltype(with_v)::value) page_load(rv, s_v, j);
        }
    };

    for (int item = 0; item < n_items; ++item) {
        qblk = item == 0 ? nqb - 1 - pair : pair;
        nt = (r + min(qblk * kBM + kBM, n) + BN - 1) / BN;
        pos = qblk * kBM + (wave >> 2) * 32 + l32;  // this lane's query column
        qabs = r + pos;
        diag = r + qblk * kBM + (wave >> 2) * 32;  // smallest query of the wave
        if (item > 0) wg_barrier();  // the previous item's output staging is done
        first_tile(flag<NW == 4>());
        // Q^T operand, all 8 dim-steps (k = 16*kb + 8*g + e)
        {
            const bool ok = active && pos < n;
            const uint16_t *qp = q + (static_cast<size_t>(row0 + (ok ? pos : 0)) * hq + h) * kHeadDim + 8 * g;
#pragma unroll
            for (int kb = 0; kb < 8; ++kb)
                qop[kb] = ok ? *reinterpret_cast<const uint4 *>(qp + 16 * kb) : make_uint4(0, 0, 0, 0);
        }
#pragma unroll
        for (int db = 0; db < 4; ++db)
#pragma unroll
            for (int i = 0; i < 16; ++i) oacc[db][i] = 0.f;
        m_run = -INFINITY;
        l_run = 0.f;
        if (item == 0) __syncthreads();  // s_bt
        __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
        wg_barrier();

        if constexpr (NW == 8) {
            // Two groups of four waves (one wave of each on every SIMD), half a
            // period apart: while one group runs its matrix phase M(t) =
            // O += V(t-1)^T P(t-1)^T, S(t) = K(t) Q^T, the other runs the
            // softmax of its previous scores on the vector ALU, so the matrix
            // cores of a SIMD stay busy through both waves' softmax.  Period t
            // (t = 0 .. nt):
            //   phase 2t:   group 0 M(t)        | group 1 softmax(t-1)
            //   phase 2t+1: group 0 softmax(t)  | group 1 M(t)
            // with a work-group barrier after each phase.  K(t+1) and V(t) are
            // loaded during period t (into the buffers K(t-1) and V(t-2) used)
            // and waited for at its end.  Row sums are plain fp32 adds: a dot
            // product instruction would wait behind the other group's MFMAs.
            const int grp = wave >> 2;
            // Each wave runs its own sequence M(0) S(0) M(1) .. S(nt-1) M(nt),
            // group 1 one phase after group 0 (a barrier ends every phase, 2nt+2
            // in all for both groups).  Group 1 issues all loads of period t
            // (K(t+1) and V(t), one page of each per wave) at the start of
            // phase 2t, its softmax phase, and waits for them at the end of
            // phase 2t+1: group 0's matrix phases issue only MFMAs and their
            // operand reads.
            const int lw = wave & 3;  // page of the tile a group-1 wave loads
            int goffp[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int row = 4 * j + (lane >> 4);
                goffp[j] = 2 * (row * kHeadDim + 8 * ((lane & 15) ^ swz(row)));
            }
            auto page_load_full = [&](__amdgpu_buffer_rsrc_t rsrc, uint16_t *dst, int j) __attribute__((always_inline)) {
                __builtin_amdgcn_raw_ptr_buffer_load_lds(
                    rsrc, reinterpret_cast<lds_void *>(reinterpret_cast<uintptr_t>(dst + (16 * lw + 4 * j) * ROW)),
                    16, goffp[j], 0, 0, 0);
            };
            // Block-table entry of page lw of tile it.  With the whole table in
            // LDS it is read one period before its loads (pg_n), so they never
            // wait for an LDS read, and taken as read (entry 0 past the
            // sequence): page_ref gives pages past the sequence no bytes and
            // tiles past the block are not loaded, so no select waits for it.
            auto table_entry = [&](int it) __attribute__((always_inline)) {
                const int p = 4 * it + lw;
                const bool ok = it < nt && p < np_seq;
                if constexpr (kTableInLds)
                    return s_bt[ok ? p - pbase : 0];
                else
                    return ok ? (p - pbase < kBtCache ? s_bt[p - pbase] : btrow[p]) : -1;
            };
            int pg_n = 0;
            PageRef ref_v{0, 0};  // page lw of tile t, whose V is loaded in period t
            auto period_loads = [&](int t) __attribute__((always_inline)) {
                PageRef ref_k;
                if constexpr (kTableInLds) {
                    ref_k = page_ref(4 * (t + 1) + lw, __builtin_amdgcn_readfirstlane(pg_n));
                    pg_n = table_entry(t + 2);
                } else {
                    ref_k = page_ref(4 * (t + 1) + lw, __builtin_amdgcn_readfirstlane(table_entry(t + 1)));
                }
                if (t + 1 < nt) {
                    const __amdgpu_buffer_rsrc_t rk = page_rsrc(kpool, ref_k);
#pragma unroll
                    for (int j = 0; j < 4; ++j) page_load_full(rk, s_k + ((t + 1) & 1) * TILE, j);
                }
                if (t < nt) {
                    const __amdgpu_buffer_rsrc_t rv = page_rsrc(vpool, ref_v);
#pragma unroll
                    for (int j = 0; j < 4; ++j) page_load_full(rv, s_v + (t & 1) * TILE, j);
                }
                ref_v = ref_k;
            };
            auto vm_wait = [&]() __attribute__((always_inline)) { __builtin_amdgcn_s_waitcnt(0x0F70); };
            if (grp == 1) {  // group 1's first phase: the loads of period 0
                ref_v = page_ref(lw, __builtin_amdgcn_readfirstlane(table_entry(0)));
                if constexpr (kTableInLds) pg_n = table_entry(1);
                period_loads(0);
                wg_barrier();
            }
            if (active) mfma_phase(flag<false>(), flag<true>(), 0, 0, [](int) {});  // M(0): S(0) = K(0) Q^T
            if (grp == 1) vm_wait();
            wg_barrier();
            for (int t = 0; t + 1 < nt; ++t) {
                if (grp == 1) period_loads(t + 1);
                if (active) softmax_phase(t);
                wg_barrier();
                if (active)  // M(t+1): O += V(t)^T P(t)^T, S(t+1) = K(t+1) Q^T
                    mfma_phase(flag<true>(), flag<true>(), (t + 1) & 1, t & 1, [](int) {});
                if (grp == 1) vm_wait();
                wg_barrier();
            }
            // the last tile: softmax(nt-1), then M(nt) = O += V(nt-1)^T P(nt-1)^T
            if (active) softmax_phase(nt - 1);
            wg_barrier();
            if (active) mfma_phase(flag<true>(), flag<false>(), 0, (nt - 1) & 1, [](int) {});
            wg_barrier();
            if (grp == 0) wg_barrier();  // group 0's last phase: none of its own work
        } else
        // Tile t+1 is loaded (into the other buffer) while tile t is processed;
        // the K and V pages of a tile are the same pages of the pool.
        for (int t = t_lo; t < (kSplit ? t_hi : nt); ++t) {
            const int u = t - t_lo;  // tile buffer parity
            const bool more = t + 1 < (kSplit ? t_hi : nt);
            const PageRef ref = more ? tile_page(t + 1) : PageRef{0, 0};
            const __amdgpu_buffer_rsrc_t rk = page_rsrc(kpool, ref), rv = page_rsrc(vpool, ref);
            uint16_t *dk = s_k + ((u + 1) & 1) * TILE;
            uint16_t *dv = s_v + ((u + 1) & 1) * TILE;
            auto load = [&](int j) __attribute__((always_inline)) {
                if (more) {
                    if (j < kJ)
                        page_load(rk, dk, j);
                    else
                        page_load(rv, dv, j - kJ);
                }
            };
            if (active) {
                mfma_phase(flag<false>(), flag<true>(), u & 1, u & 1, load);
                softmax_phase(t);
                mfma_phase(flag<true>(), flag<false>(), u & 1, u & 1, [](int) {});
            } else {
#pragma unroll
                for (int j = 0; j < 2 * kJ; ++j) load(j);
            }
            __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): this wave's direct loads landed
            wg_barrier();
        }

        if constexpr (kSplit) {
            if (n_pieces > 1) {
                // ---- this piece's partial: (m, l) and the unnormalised O of
                // every row, fp32.  The wave's 32 x 128 tile (16 KiB; waves 0-1
                // in the K buffers, 2-3 in the V buffers) is staged in LDS so
                // every store writes whole 512-byte rows; row q holds its
                // 16-byte chunk c (dims 4c..4c+3) at chunk c ^ (q % 32).
                const float lt = l_run + __shfl_xor(l_run, 32);
                char *st = reinterpret_cast<char *>(wave < 2 ? s_k : s_v) + (wave & 1) * (32 * 512);
#pragma unroll
                for (int db = 0; db < 4; ++db)
#pragma unroll
                    for (int i4 = 0; i4 < 4; ++i4) {
                        const int c = 8 * db + 2 * i4 + g;
                        *reinterpret_cast<float4 *>(st + l32 * 512 + 16 * (c ^ l32)) =
                            make_float4(oacc[db][4 * i4 + 0], oacc[db][4 * i4 + 1], oacc[db][4 * i4 + 2],
                                        oacc[db][4 * i4 + 3]);
                    }
                if (active) {
                    const size_t slot = static_cast<size_t>(sp.piece) * sp.rows + row0;
#pragma unroll
                    for (int j = 0; j < 16; ++j) {
                        const int row = 2 * j + (lane >> 5), c = lane & 31;
                        const float4 v = *reinterpret_cast<const float4 *>(st + row * 512 + 16 * (c ^ row));
                        const int prow = qblk * kBM + row;
                        if (prow < n)
                            *reinterpret_cast<float4 *>(sp.o + ((slot + prow) * hq + h) * kHeadDim + 4 * c) = v;
                    }
                    if (g == 0 && pos < n) sp.ml[(slot + pos) * hq + h] = make_float2(m_run, lt);
                }
                continue;
            }
        }
        // ---- normalise and write O[pos][h][d].  The wave's 32 x 128 tile is
        // staged in LDS (the K/V buffers are free now) so that every store
        // writes 16 bytes per lane and four whole 256-byte rows per
        // instruction.  Row q of the staged tile holds its 16-byte chunk c at
        // chunk c ^ (q % 16).
        const float lt = l_run + __shfl_xor(l_run, 32);
        const float inv = 1.f / lt;
        char *st = reinterpret_cast<char *>((wave < 4 ? s_k : s_v) + (wave & 3) * (32 * ROW));
#pragma unroll
        for (int db = 0; db < 4; ++db)
#pragma unroll
            for (int i4 = 0; i4 < 4; ++i4) {
                const int c = 4 * db + i4;
                *reinterpret_cast<uint2 *>(st + l32 * 256 + 16 * (c ^ (l32 & 15)) + 8 * g) =
                    make_uint2(cvt2(oacc[db][4 * i4 + 0] * inv, oacc[db][4 * i4 + 1] * inv),
                               cvt2(oacc[db][4 * i4 + 2] * inv, oacc[db][4 * i4 + 3] * inv));
            }
        if (active) {
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const int row = 4 * j + (lane >> 4), c = lane & 15;
                const uint4 v = *reinterpret_cast<const uint4 *>(st + row * 256 + 16 * (c ^ (row & 15)));
                const int prow = qblk * kBM + (wave >> 2) * 32 + row;
                if (prow < n)
                    *reinterpret_cast<uint4 *>(out + (static_cast<size_t>(row0 + prow) * hq + h) * kHeadDim + 8 * c) = v;
            }
        }
    }
}


}  // namespace pf
}  // namespace
