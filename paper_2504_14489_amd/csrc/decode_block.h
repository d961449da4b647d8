// Device body of the split-K decode attention (one work unit), shared by
// the decode kernel and the fused prefill + decode kernel.
//
// Decode is memory-bound (paper Sec. 2.2: the decode phase is
// memory-intensive; Sec. 3.3, Table "tab:theory_cost": O(d^2 + (r+1) d)), so
// the design goal is streaming every K/V byte of the batch from HBM exactly
// once with enough bytes in flight; arithmetic is kept off the vector ALU.
//
// Work-group = (sequence b, kv head, chunk of CH consecutive pages), 4 waves.
// The split depends only on the sequence lengths (never on page ids), so a
// result does not change when pages are renumbered.
//
// Each wave streams its own pages of the chunk two at a time (a "pair"), with
// the next pair's loads in flight while the current pair is computed.  K and
// V rows are loaded whole (each instruction reads four 256-byte rows, so no
// cache line is requested twice) with streaming loads that leave nothing in
// the caches for the other partition's kernel to lose, and go to per-wave LDS
// buffers as loaded (16-byte row-major stores):
//   * K comes back in the A-operand layout of a 16x16x32 bf16 MFMA (one page
//     = 16 tokens x 32 dims per step), B = Q^T of the kv head's G query heads
//     (columns >= G are zero): S^T[token][head].
//   * V comes back through the transposing LDS read as the A operand of a
//     second MFMA, O^T[d][head] += V^T[d][token] P^T[token][head]; P^T is the
//     S^T accumulator itself, converted to bf16.
//   * online softmax per pair in base 2; the reference maximum moves only
//     when a column's maximum grows by more than 2^8 (O and l are then
//     rescaled), which the result O / l does not depend on.
// The 4 waves' (m, l, O) are merged in LDS at the end; a sequence that fits
// one chunk writes its bf16 output directly, otherwise the chunk's partial goes
// to the workspace and the pieces of each (sequence, kv head) are merged with
// the log-sum-exp identity
//   M = max m_s,  O = sum 2^(m_s - M) o_s / sum 2^(m_s - M) l_s
// by the work-group that finishes the segment's last piece (balanced split)
// or by the combine kernel (fixed chunks).
#pragma once
#include "mw_internal.h"

namespace {
namespace dk {

using namespace mw;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
constexpr int kPair = 2;                      // pages per wave step
constexpr int VSTR = 144;                     // LDS V row stride (bf16): conflict-free transposing reads
constexpr int KSTR = 136;                     // LDS K row stride (bf16): conflict-free 16-byte reads
constexpr int kVBufElems = 16 * kPair * VSTR; // one wave's V buffer
constexpr int kKBufElems = 16 * kPair * KSTR; // one wave's K buffer
constexpr int kWaveBufElems = kVBufElems + kKBufElems;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kRescaleLog2 = 8.f;
// chunk_pages = 0: the largest of 128, 64, 32 pages that still gives at least
// kAutoMinUnits work-groups (longer chunks amortise each work-group's set-up
// and merge; enough work-groups keep every CU of a partition streaming)
constexpr int kAutoChunks[3] = {128, 64, 32};
constexpr int64_t kAutoMinUnits = 1024;

__device__ inline uint16_t to_bf16(float f) { return __builtin_bit_cast(uint16_t, static_cast<__bf16>(f)); }
__device__ inline uint32_t cvt2(float a, float b) {
    bf16x2 v;
    v[0] = static_cast<__bf16>(a);
    v[1] = static_cast<__bf16>(b);
    return __builtin_bit_cast(uint32_t, v);
}
__device__ inline uint4 sel4(bool ok, uint4 v) {
    return make_uint4(ok ? v.x : 0u, ok ? v.y : 0u, ok ? v.z : 0u, ok ? v.w : 0u);
}
__device__ inline i16x4 lds_read_tr(const uint16_t *p) {
    return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        reinterpret_cast<__attribute__((address_space(3))) i16x4 *>(reinterpret_cast<uintptr_t>(p)));
}

__device__ inline int chunks_of(int L, int ch_pages, int bt_stride) {
    if (L <= 0) return 0;
    int np = (L + kPageSize - 1) / kPageSize;
    np = np < bt_stride ? np : bt_stride;
    return (np + ch_pages - 1) / ch_pages;
}

// Wave-level search for the sequence b and chunk c holding global chunk ci
// (every wave runs it; no barrier).  Returns false if ci is past the end.
__device__ bool locate_chunk(const int32_t *__restrict__ seq_lens, int batch, int ch_pages, int bt_stride,
                             int ci, int &b_out, int &c_out, int &nch_out, int &first_out) {
    const int lane = threadIdx.x & 63;
    int running = 0;
    for (int base = 0; base < batch; base += 64) {
        const int bb = base + lane;
        const int n = bb < batch ? chunks_of(seq_lens[bb], ch_pages, bt_stride) : 0;
        int x = n;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const int y = __shfl_up(x, off);
            if (lane >= off) x += y;
        }
        const int incl = running + x, excl = incl - n;
        const uint64_t hit = __builtin_amdgcn_ballot_w64(bb < batch && ci >= excl && ci < incl);
        if (hit) {
            const int src = __builtin_ctzll(hit);
            first_out = __shfl(excl, src);
            b_out = base + src;
            c_out = ci - first_out;
            nch_out = __shfl(n, src);
            return true;
        }
        running = __shfl(incl, 63);
    }
    return false;
}

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
// Streaming load: the line is not kept in the caches (decode reads each byte
// of K/V once), so the other partition's working set stays there.
__device__ inline uint4 load_stream(const uint16_t *p) {
    return __builtin_bit_cast(uint4, __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(p)));
}

struct PairRegs {
    uint4 k[kPair][4];  // K rows as loaded: token 4i + lane/16, dims 8(lane%16) + 0..7
    uint4 v[kPair][4];  // V rows: token 4i + lane/16, dims 8(lane%16) + 0..7
    bool ok[kPair];
};

__device__ inline void pair_load(PairRegs &pr, const uint16_t *__restrict__ kpool,
                                 const uint16_t *__restrict__ vpool, const int32_t *__restrict__ btrow,
                                 int p0, int p_end, int hkv, int kvh, int num_pages) {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int j = 0; j < kPair; ++j) {
        const int p = p0 + j;
        const int page = btrow[p < p_end ? p : p0];
        pr.ok[j] = p < p_end && page >= 0 && page < num_pages;
        const size_t base = (static_cast<size_t>(pr.ok[j] ? page : 0) * hkv + kvh) * (kPageSize * kHeadDim);
        // whole 256-byte rows per instruction (four rows each), so no cache
        // line is requested by two instructions
#pragma unroll
        for (int i = 0; i < 4; ++i)
            pr.k[j][i] = load_stream(kpool + base + (4 * i + (lane >> 4)) * kHeadDim + 8 * (lane & 15));
#pragma unroll
        for (int i = 0; i < 4; ++i)
            pr.v[j][i] = load_stream(vpool + base + (4 * i + (lane >> 4)) * kHeadDim + 8 * (lane & 15));
    }
}

// Pages [p_begin, p_end) of sequence b (length L, block-table row btrow),
// kv head kvh, on 4 waves; tid = thread index within them (0..255); s_v,
// s_m, s_l are their LDS.  The merged result is written as the bf16 output
// (direct) or as the fp32 partial (O, (m, l)) of workspace slot `slot`.
// active = false (uniform): nothing is read or written, but both work-group
// barriers are still taken.
__device__ __forceinline__ void
decode_pages(const uint16_t *__restrict__ kpool, const uint16_t *__restrict__ vpool,
             const uint16_t *__restrict__ q, uint16_t *__restrict__ out, const int32_t *__restrict__ btrow,
             float *__restrict__ ws_o, float2 *__restrict__ ws_ml, int b, int L, int hkv, int kvh, int group,
             int num_pages, float scale_log2, int p_begin, int p_end, bool active, bool direct, int64_t slot,
             int tid, uint16_t *s_v, float (*s_m)[16], float (*s_l)[16]) {
    const int lane = tid & 63, wave = tid >> 6;
    const int col = lane & 15, grp = lane >> 4;
    if (!active) p_end = p_begin;
    const int hq = hkv * group;

    // Q^T operand: column `col` is query head kvh*group + col
    uint4 qop[4];
    {
        const bool hv = col < group;
        const uint16_t *qp = q + (static_cast<size_t>(b) * hq + kvh * group + (hv ? col : 0)) * kHeadDim + 8 * grp;
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
            qop[kb] = hv ? *reinterpret_cast<const uint4 *>(qp + 32 * kb) : make_uint4(0, 0, 0, 0);
    }

    f32x4 oacc[8];  // O^T[d = 16db + 4grp + i][head = col]
#pragma unroll
    for (int db = 0; db < 8; ++db) oacc[db] = f32x4{0.f, 0.f, 0.f, 0.f};
    float m_run = -INFINITY, l_run = 0.f;

    uint16_t *vbuf = s_v + wave * kWaveBufElems;
    uint16_t *kbuf = vbuf + kVBufElems;
    // K operand reads: lane l reads row l%16 of each page, 16-byte chunk 4kb + l/16
    const uint16_t *krd = kbuf + col * KSTR + 8 * grp;
    // transposing-read source: lane s of 16-lane group g -> row 4g + s/4 (+16 for
    // the second page), dims 4(s%4) (+16 db)
    const uint16_t *vtr = vbuf + (4 * grp + (col >> 2)) * VSTR + 4 * (col & 3);

    // this wave's pairs: pages p_begin + 2*(wave + 4*j) + {0, 1}
    const int pstart = p_begin + kPair * wave;
    const int pstep = kPair * kWaves;
    PairRegs pr;
    if (pstart < p_end) pair_load(pr, kpool, vpool, btrow, pstart, p_end, hkv, kvh, num_pages);
    for (int p0 = pstart; p0 < p_end; p0 += pstep) {
        bool ok[kPair];
#pragma unroll
        for (int j = 0; j < kPair; ++j) ok[j] = pr.ok[j];
        // K and V of this pair -> LDS as loaded, with V rows of an absent page
        // or past the sequence's end as zeros (a masked key has p = 0, but 0
        // times a NaN or Inf in a slack slot would not be 0); the scores of
        // those keys are masked below
#pragma unroll
        for (int j = 0; j < kPair; ++j)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                *reinterpret_cast<uint4 *>(kbuf + (16 * j + 4 * i + grp) * KSTR + 8 * col) = pr.k[j][i];
                *reinterpret_cast<uint4 *>(vbuf + (16 * j + 4 * i + grp) * VSTR + 8 * col) =
                    sel4(pr.ok[j] && (p0 + j) * kPageSize + 4 * i + grp < L, pr.v[j][i]);
            }
        // next pair's loads go out while this pair is computed
        const int pn = p0 + pstep;
        if (pn < p_end) pair_load(pr, kpool, vpool, btrow, pn, p_end, hkv, kvh, num_pages);
        // S^T = K Q^T on the matrix core, K read back in the operand layout
        f32x4 sc[kPair];
#pragma unroll
        for (int j = 0; j < kPair; ++j) {
            sc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int kb = 0; kb < 4; ++kb) {
                const uint4 a = *reinterpret_cast<const uint4 *>(krd + 16 * j * KSTR + 32 * kb);
                sc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                                __builtin_bit_cast(bf16x8, qop[kb]), sc[j], 0, 0, 0);
            }
        }

        // mask keys past the sequence or on an absent page, then the pair's
        // maximum per head
        float mx = -INFINITY;
#pragma unroll
        for (int j = 0; j < kPair; ++j)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int tok = (p0 + j) * kPageSize + 4 * grp + i;
                const float v = (ok[j] && tok < L) ? sc[j][i] * scale_log2 : -INFINITY;
                sc[j][i] = v;
                mx = fmaxf(mx, v);
            }
        mx = fmaxf(mx, __shfl_xor(mx, 16));
        mx = fmaxf(mx, __shfl_xor(mx, 32));
        if (__builtin_amdgcn_ballot_w64(mx > m_run + kRescaleLog2) != 0) {
            const float m_new = fmaxf(m_run, mx);
            const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
            m_run = m_new;
            l_run *= alpha;
#pragma unroll
            for (int db = 0; db < 8; ++db) oacc[db] *= alpha;
        }
        float p[kPair][4];
#pragma unroll
        for (int j = 0; j < kPair; ++j)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                p[j][i] = __builtin_amdgcn_exp2f(sc[j][i] - m_run);
                l_run += p[j][i];
            }
        // P^T operand: k-slot e < 4 is token 4grp+e of page 0, e >= 4 token
        // 16 + 4grp + e-4 of page 1 -- the V^T reads below use the same order
        const uint4 pop = make_uint4(cvt2(p[0][0], p[0][1]), cvt2(p[0][2], p[0][3]),
                                     cvt2(p[1][0], p[1][1]), cvt2(p[1][2], p[1][3]));
#pragma unroll
        for (int db = 0; db < 8; ++db) {
            const i16x4 lo = lds_read_tr(vtr + 16 * db);
            const i16x4 hi = lds_read_tr(vtr + 16 * VSTR + 16 * db);
            const bf16x8 a = __builtin_bit_cast(
                bf16x8, make_uint4(__builtin_bit_cast(uint2, lo).x, __builtin_bit_cast(uint2, lo).y,
                                   __builtin_bit_cast(uint2, hi).x, __builtin_bit_cast(uint2, hi).y));
            oacc[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, __builtin_bit_cast(bf16x8, pop), oacc[db], 0, 0, 0);
        }
    }

    // ---- merge the 4 waves: per-head (m, l) and O^T through LDS
    l_run += __shfl_xor(l_run, 16);
    l_run += __shfl_xor(l_run, 32);
    if (grp == 0) {
        s_m[wave][col] = m_run;
        s_l[wave][col] = l_run;
    }
    __syncthreads();  // every wave is done with its V buffer: reuse it for O^T
    float *s_o = reinterpret_cast<float *>(s_v);  // [kWaves][128 d][16 heads]
#pragma unroll
    for (int db = 0; db < 8; ++db)
#pragma unroll
        for (int i = 0; i < 4; ++i) s_o[(wave * kHeadDim + 16 * db + 4 * grp + i) * 16 + col] = oacc[db][i];
    __syncthreads();
    for (int idx = tid; active && idx < group * kHeadDim; idx += kThreads) {
        const int h = idx / kHeadDim, d = idx % kHeadDim;
        float M = -INFINITY;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) M = fmaxf(M, s_m[w][h]);
        float lsum = 0.f, o = 0.f;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) {
            const float mw = s_m[w][h];
            const float wt = mw == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(mw - M);  // waves without pages
            lsum += wt * s_l[w][h];
            o += wt * s_o[(w * kHeadDim + d) * 16 + h];
        }
        if (direct) {
            out[(static_cast<size_t>(b) * hq + kvh * group + h) * kHeadDim + d] = to_bf16(o / lsum);
        } else {
            // device-scope stores (through the L2 of this XCD): the piece may be
            // merged by a work-group on another XCD without a cache writeback
            __hip_atomic_store(&ws_o[(static_cast<size_t>(slot) * group + h) * kHeadDim + d], o, __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
            if (d == 0)
                __hip_atomic_store(reinterpret_cast<unsigned long long *>(&ws_ml[static_cast<size_t>(slot) * group + h]),
                                   __builtin_bit_cast(unsigned long long, make_float2(M, lsum)), __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
        }
    }
}

// One (sequence, kv head, chunk) work unit of the fixed-chunk split: unit u
// is chunk u / hkv of the batch's chunks in order, kv head u % hkv.  A
// sequence of one chunk is written directly; otherwise the chunk's partial
// goes to slot u and the sequence's first chunk index to ws_cbase[b].
// kGuarded: the caller runs other work in the same work-group, so a unit
// past the end does nothing but still takes the two work-group barriers.
template <bool kGuarded>
__device__ __forceinline__ void
decode_unit(const uint16_t *__restrict__ kpool, const uint16_t *__restrict__ vpool,
            const uint16_t *__restrict__ q, uint16_t *__restrict__ out, const int32_t *__restrict__ seq_lens,
            const int32_t *__restrict__ bt, int bt_stride, float *__restrict__ ws_o, float2 *__restrict__ ws_ml,
            int32_t *__restrict__ ws_cbase, int batch, int hkv, int group, int num_pages, float scale_log2,
            int ch_pages, int u, int tid, uint16_t *s_v, float (*s_m)[16], float (*s_l)[16]) {
    const int kvh = u % hkv;
    int b = 0, c = 0, nch = 0, first = 0;
    const bool found = locate_chunk(seq_lens, batch, ch_pages, bt_stride, u / hkv, b, c, nch, first);
    // more units than the device lengths give (uniform over the 4 waves): a
    // kernel of its own returns; a fused work-group still takes both barriers
    if constexpr (!kGuarded) {
        if (!found) return;
    }
    const int L = min(seq_lens[b], bt_stride * kPageSize);
    const int np_b = (L + kPageSize - 1) / kPageSize;
    decode_pages(kpool, vpool, q, out, bt + static_cast<size_t>(b) * bt_stride, ws_o, ws_ml, b, L, hkv, kvh,
                 group, num_pages, scale_log2, c * ch_pages, min((c + 1) * ch_pages, np_b), found, nch == 1, u,
                 tid, s_v, s_m, s_l);
    if (found && c == 0 && kvh == 0 && tid == 0) ws_cbase[b] = first;
}

// Wave-level search for the sequence b whose kv-head segments hold global
// page g of the balanced split (segments in the order (b, kv head), each of
// the sequence's page count, rounded up to a multiple of `align` when it is
// not 0); base_out = hkv * (such counts of the sequences < b).  Returns false
// if g is past the end.
__device__ bool locate_page(const int32_t *__restrict__ seq_lens, int batch, int bt_stride, int hkv, int64_t align,
                            int64_t g, int &b_out, int64_t &base_out) {
    const int lane = threadIdx.x & 63;
    int64_t running = 0;
    for (int base = 0; base < batch; base += 64) {
        const int bb = base + lane;
        int64_t np = bb < batch ? chunks_of(seq_lens[bb], 1, bt_stride) : 0;
        if (align > 0) np = (np + align - 1) / align * align;
        const int64_t n = static_cast<int64_t>(hkv) * np;
        int64_t x = n;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const int64_t y = __shfl_up(x, off);
            if (lane >= off) x += y;
        }
        const int64_t incl = running + x, excl = incl - n;
        const uint64_t hit = __builtin_amdgcn_ballot_w64(bb < batch && g >= excl && g < incl);
        if (hit) {
            const int src = __builtin_ctzll(hit);
            base_out = __shfl(excl, src);
            b_out = base + src;
            return true;
        }
        running = __shfl(incl, 63);
    }
    return false;
}

// Merges the pieces j = 0 .. nch-1 of segment (b, kv head), piece j's partial
// in workspace slot first + j * stride, into the bf16 output (the combine
// kernel).  One pass over the pieces with a running maximum; each thread
// merges two outputs (h, d), and the (m, l) and o of 8 pieces of both are
// loaded together, so a short segment costs one round of loads.
__device__ __forceinline__ void
merge_pieces(uint16_t *__restrict__ out, const float *__restrict__ ws_o, const float2 *__restrict__ ws_ml,
             int64_t first, int64_t stride, int nch, int b, int hkv, int kvh, int group, int tid) {
    const int hq = hkv * group;
    const int n_out = group * kHeadDim;
    for (int i0 = tid; i0 < n_out; i0 += 2 * kThreads) {
        const int idx[2] = {i0, i0 + kThreads};
        float M[2] = {-INFINITY, -INFINITY}, lsum[2] = {0.f, 0.f}, osum[2] = {0.f, 0.f};
        for (int s0 = 0; s0 < nch; s0 += 8) {
            float2 ml[2][8];
            float o[2][8];
#pragma unroll
            for (int k = 0; k < 2; ++k)
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    const bool in = s0 + j < nch && idx[k] < n_out;
                    const int h = in ? idx[k] / kHeadDim : 0, d = idx[k] % kHeadDim;
                    const size_t uu = static_cast<size_t>(first + (s0 + j) * stride) * group + h;
                    ml[k][j] = in ? ws_ml[uu] : make_float2(-INFINITY, 0.f);
                    o[k][j] = in ? ws_o[uu * kHeadDim + d] : 0.f;
                }
#pragma unroll
            for (int k = 0; k < 2; ++k)
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    if (!(ml[k][j].y > 0.f)) continue;  // a piece without keys contributes nothing
                    const float mn = fmaxf(M[k], ml[k][j].x);
                    const float a = __builtin_amdgcn_exp2f(M[k] - mn), w = __builtin_amdgcn_exp2f(ml[k][j].x - mn);
                    lsum[k] = lsum[k] * a + w * ml[k][j].y;
                    osum[k] = osum[k] * a + w * o[k][j];
                    M[k] = mn;
                }
        }
#pragma unroll
        for (int k = 0; k < 2; ++k)
            if (idx[k] < n_out) {
                const int h = idx[k] / kHeadDim, d = idx[k] % kHeadDim;
                out[(static_cast<size_t>(b) * hq + kvh * group + h) * kHeadDim + d] = to_bf16(osum[k] / lsum[k]);
            }
    }
}

// Merge of one balanced-split segment in the work-group that finished its
// last piece; pieces j = 0 .. nch-1 in slots first + j, read at device scope
// (they were written in this kernel, possibly on other XCDs).  First the
// pieces' (m, l), which lie together in the workspace, all go to LDS and one
// wave per head reduces the maximum M and the denominator
// sum_j 2^(m_j - M) l_j; then each wave streams the partial O of one head
// at a time, two outputs per lane with 8 pieces of both in flight, weighting
// each piece by 2^(m_j - M).
// s_ml holds nch * group entries (at most kMergeMaxEntries).
constexpr int kMergeMaxEntries = kWaves * kWaveBufElems * 2 / 8;
constexpr int kBufferFormat32 = 0x00020000;  // buffer descriptor word 3: 32-bit data format
constexpr int kLoadDeviceScope = 16;         // buffer load cache policy: device scope
__device__ __forceinline__ void
merge_segment(uint16_t *__restrict__ out, const float *__restrict__ ws_o, const float2 *__restrict__ ws_ml,
              int64_t first, int nch, int b, int hkv, int kvh, int group, int tid, float2 *s_ml, float *s_M,
              float *s_L) {
    const int lane = tid & 63, wave = tid >> 6;
    const int n_ml = nch * group;
    unsigned long long *ml_src = reinterpret_cast<unsigned long long *>(const_cast<float2 *>(ws_ml)) + first * group;
    for (int e = tid; e < n_ml; e += kThreads)
        s_ml[e] = __builtin_bit_cast(float2, __hip_atomic_load(ml_src + e, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
    __syncthreads();
    for (int h = wave; h < group; h += kWaves) {
        float M = -INFINITY;
        for (int j = lane; j < nch; j += 64) {
            const float2 v = s_ml[j * group + h];
            if (v.y > 0.f) M = fmaxf(M, v.x);  // a piece without keys contributes nothing
        }
#pragma unroll
        for (int sh = 32; sh >= 1; sh >>= 1) M = fmaxf(M, __shfl_xor(M, sh));
        float L = 0.f;
        for (int j = lane; j < nch; j += 64) {
            const float2 v = s_ml[j * group + h];
            if (v.y > 0.f) L += __builtin_amdgcn_exp2f(v.x - M) * v.y;
        }
#pragma unroll
        for (int sh = 32; sh >= 1; sh >>= 1) L += __shfl_xor(L, sh);
        if (lane == 0) {
            s_M[h] = M;
            s_L[h] = L;
        }
    }
    __syncthreads();
    const int hq = hkv * group;
    const int n_out = group * kHeadDim;
    // the pieces' partial O through a buffer resource: one offset register per
    // output, the piece's offset in the scalar operand, device-scope loads.
    // One wave per head, each lane two of its outputs, so a piece's weight is
    // one broadcast LDS read for both.
    const __amdgpu_buffer_rsrc_t r_o =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<float *>(ws_o) + static_cast<size_t>(first) * n_out, 0,
                                          nch * n_out * 4, kBufferFormat32);
    for (int h = wave; h < group; h += kWaves) {
        const float M = s_M[h];
        float acc0 = 0.f, acc1 = 0.f;
        for (int j0 = 0; j0 < nch; j0 += 8) {
            float o0[8], o1[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const bool in = j0 + j < nch;
                const int off = 4 * (j0 + j) * n_out;
                o0[j] = in ? __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                                                           r_o, 4 * (h * kHeadDim + lane), off, kLoadDeviceScope))
                           : 0.f;
                o1[j] = in ? __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                                                           r_o, 4 * (h * kHeadDim + 64 + lane), off, kLoadDeviceScope))
                           : 0.f;
            }
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                if (j0 + j >= nch) break;
                const float2 v = s_ml[(j0 + j) * group + h];
                const float w = v.y > 0.f ? __builtin_amdgcn_exp2f(v.x - M) : 0.f;
                acc0 += w * o0[j];
                acc1 += w * o1[j];
            }
        }
        const float inv = 1.f / s_L[h];
        uint16_t *orow = out + (static_cast<size_t>(b) * hq + kvh * group + h) * kHeadDim;
        orow[lane] = to_bf16(acc0 * inv);
        orow[64 + lane] = to_bf16(acc1 * inv);
    }
}

// A work-group that has written its pieces of split segments (at most two:
// the unit's first and last) marks them done in their flags (this call's
// tag) and reads the segments' other flags, both segments in one round; a
// work-group that finds every piece of a segment done merges the segment and
// clears its flags.  The work-group that marks last always finds them all;
// two that finish together may both merge, writing the same bits.  Pieces
// and flags are written and read with device-scope stores and loads
// (coherent across the XCDs' L2 caches), and each wave waits for its stores
// to complete before the next step; release/acquire fences would instead
// write back and invalidate the whole L2 of the XCD for every work-group, and
// one counter per segment would serialise the pieces' atomics.  A flag from an
// earlier call shows another tag (tags are never 0, the cleared value), so
// the workspace needs no initialisation, and a replay of the same launch (same
// tag) finds the flags cleared.  No work-group waits for another.
__device__ __forceinline__ void
finish_segments(uint16_t *__restrict__ out, const float *__restrict__ ws_o, const float2 *__restrict__ ws_ml,
                uint32_t *__restrict__ flags, uint32_t tag, int npend, const int64_t *first, const int *nch,
                const int64_t *self, const int *sb, const int *skvh, int64_t slots, int hkv, int group, int tid,
                float2 *s_ml, float *s_M, float *s_L) {
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // this wave's piece stores are complete
    __syncthreads();
    if (tid == 0) {
        for (int i = 0; i < npend; ++i)
            if (self[i] >= 0 && self[i] < slots)
                __hip_atomic_store(flags + self[i], tag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    }
    __syncthreads();
    // both segments' flags in one round of loads; device lengths that
    // disagree with the host's must not lead outside the workspace
    bool ok[2], done[2] = {true, true};
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        ok[i] = i < npend && first[i] >= 0 && first[i] + nch[i] - 1 < slots && nch[i] * group <= kMergeMaxEntries;
        for (int j = tid; ok[i] && j < nch[i]; j += kThreads)
            done[i] &= __hip_atomic_load(flags + first[i] + j, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == tag;
    }
    const bool all0 = __syncthreads_and(ok[0] && done[0]);
    const bool all1 = __syncthreads_and(ok[1] && done[1]);
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        if (!(i == 0 ? all0 : all1)) continue;
        for (int j = tid; j < nch[i]; j += kThreads)
            __hip_atomic_store(flags + first[i] + j, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (i == 1 && all0) __syncthreads();  // the first merge is done with the LDS
        merge_segment(out, ws_o, ws_ml, first[i], nch[i], sb[i], hkv, skvh[i], group, tid, s_ml, s_M, s_L);
    }
}

// One unit of the balanced split: global pages [u R, min((u + 1) R, total))
// of the (sequence, kv head) segments in order, which may cross segment
// boundaries; with `aligned`, every segment is padded to a multiple of R
// pages (the padding holds no pages), so a unit holds one piece of one
// segment.  Each segment piece is merged on its own: a segment the unit
// holds whole is written directly, a piece of a longer segment goes to slot
// u + s (s = b hkv + kv head) with its done flag in `flags` at the same
// index, and the work-group that finds every piece of the segment done
// merges them (those of units P / R .. (P + pages(b) - 1) / R, P the
// segment's first global page).
// Not for fused work-groups: the number of barriers depends on the unit.
__device__ __forceinline__ void
decode_span(const uint16_t *__restrict__ kpool, const uint16_t *__restrict__ vpool,
            const uint16_t *__restrict__ q, uint16_t *__restrict__ out, const int32_t *__restrict__ seq_lens,
            const int32_t *__restrict__ bt, int bt_stride, float *__restrict__ ws_o, float2 *__restrict__ ws_ml,
            uint32_t *__restrict__ flags, uint32_t tag, int64_t slots, int batch, int hkv, int group,
            int num_pages, float scale_log2, int64_t per_unit, int64_t total, bool aligned, int u, int tid,
            uint16_t *s_v, float (*s_m)[16], float (*s_l)[16]) {
    int64_t g = static_cast<int64_t>(u) * per_unit;
    const int64_t g_end = min(g + per_unit, total);
    int b = 0;
    int64_t base_b = 0;
    const int64_t align = aligned ? per_unit : 0;
    if (g >= g_end || !locate_page(seq_lens, batch, bt_stride, hkv, align, g, b, base_b)) return;
    int L = min(seq_lens[b], bt_stride * kPageSize);
    int np_b = (L + kPageSize - 1) / kPageSize;
    // the segment's extent in the split's page numbering (padded when aligned)
    auto extent = [&](int np) { return aligned ? static_cast<int>((np + align - 1) / align * align) : np; };
    int nv_b = extent(np_b);
    int kvh = static_cast<int>((g - base_b) / nv_b);
    int off = static_cast<int>((g - base_b) % nv_b);
    // the unit's pieces of split segments (only its first and last piece can
    // be): counted in and merged after all its pages, when none of the page
    // loop's registers are live any more
    int pend_b[2] = {0, 0}, pend_kvh[2] = {0, 0}, pend_nch[2] = {0, 0}, npend = 0;
    int64_t pend_first[2] = {0, 0}, pend_self[2] = {0, 0};
    for (bool first = true; g < g_end; first = false) {
        // n pages of the split's numbering, of which those below np_b exist
        const int n = static_cast<int>(min(static_cast<int64_t>(nv_b - off), g_end - g));
        const int p_end = min(off + n, np_b);
        if (!first) __syncthreads();  // the previous piece is done with the LDS
        const bool whole = off == 0 && p_end == np_b && n == nv_b;
        const int64_t seg = static_cast<int64_t>(b) * hkv + kvh;
        decode_pages(kpool, vpool, q, out, bt + static_cast<size_t>(b) * bt_stride, ws_o, ws_ml, b, L, hkv, kvh,
                     group, num_pages, scale_log2, off, p_end, true, whole, static_cast<int64_t>(u) + seg, tid, s_v,
                     s_m, s_l);
        if (!whole && npend < 2) {
            const int64_t p0 = base_b + static_cast<int64_t>(kvh) * nv_b;
            const int64_t u0 = p0 / per_unit, u1 = (p0 + nv_b - 1) / per_unit;
            pend_b[npend] = b;
            pend_kvh[npend] = kvh;
            pend_first[npend] = u0 + seg;
            pend_self[npend] = static_cast<int64_t>(u) + seg;
            pend_nch[npend] = static_cast<int>(u1 - u0 + 1);
            ++npend;
        }
        g += n;
        off = 0;
        if (++kvh == hkv) {
            kvh = 0;
            base_b += static_cast<int64_t>(hkv) * nv_b;
            if (++b >= batch) break;
            L = min(seq_lens[b], bt_stride * kPageSize);
            np_b = (L + kPageSize - 1) / kPageSize;
            nv_b = extent(np_b);
            if (np_b == 0) break;  // device lengths that disagree with the host's
        }
    }
    if (npend > 0)
        finish_segments(out, ws_o, ws_ml, flags, tag, npend, pend_first, pend_nch, pend_self, pend_b, pend_kvh, slots,
                        hkv, group, tid, reinterpret_cast<float2 *>(s_v), s_m[0], s_l[0]);
}

}  // namespace dk
}  // namespace
