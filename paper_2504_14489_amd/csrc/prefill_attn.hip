// Causal prefill attention of a chunk of new tokens over its cached prefix.
//
// Prefill is compute-bound (paper Sec. 2.2; Sec. 3.3, Table
// "tab:theory_cost": O(n d^2 + L n d) with L = r + n), so both contractions
// run on the bf16 matrix cores (fp32 accumulate); the vector ALU, which also
// has to run the softmax, is kept to the few instructions per score that the
// softmax itself needs.
//
// Work-group = 8 waves = 64 query positions x 4 query heads of one kv head;
// wave w owns head (w % 4) of the group and positions 32*(w / 4) .. +31, so
// every K/V tile staged in LDS serves 4 heads x 64 positions.  Two waves share
// each SIMD; each wave's state (Q^T, S, O, P) stays in VGPRs.
// Key tiles of 64 keys = 4 pages go from HBM straight into LDS with the direct
// global-to-LDS loads (no staging registers): each wave moves half a page of K
// and of V per tile (4 instructions of 4 rows x 256 B), double-buffered.  Rows
// are 256 B with their 16-byte chunks permuted by XOR with
// swz(r) = 4(r%4) ^ (r/4)%4, which makes both the 16-byte K operand reads and
// the transposing V reads bank-conflict free; the permutation is applied on
// the HBM side of each load, and every lane's LDS read offsets are computed
// once before the loop.
// Per tile and wave:
//   S^T[key][q] = K Q^T      32x32x16 MFMA; A = K rows from LDS, B = Q^T held
//                            in registers for the whole kernel
//   online softmax in base 2 (scores scaled by scale*log2 e inside one FMA);
//   the causal mask is applied only on tiles that cross the diagonal; row sums
//   are taken from the bf16 probabilities with packed dot products
//   O^T[d][q] += V^T P^T     32x32x16 MFMA; A = V^T gathered by the LDS
//                            transposing read (ds_read_b64_tr_b16), B = P^T taken
//                            straight from the S^T accumulators as bf16
// The running maximum moves only when a column's tile maximum exceeds it by
// more than 2^8 (O and l are then rescaled); O / l does not depend on the
// reference maximum.
// Causal position: query row i of a sequence with prefix r sees keys
// 0 .. r + i (bottom-right alignment; a chunk reads every earlier chunk's KV).
#include "mw_internal.h"

using namespace mw;

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kWaves = 8;
constexpr int kThreads = 64 * kWaves;
constexpr int BM = 64;                       // query positions per work-group
constexpr int BN = 64;                       // keys per tile
constexpr int ROW = kHeadDim;                // tile row = one key, 128 bf16 (256 B)
constexpr int TILE = BN * ROW;               // one K or V tile, bf16 elements
constexpr int kBtCache = 4096;               // block-table entries staged in LDS
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kRescaleLog2 = 8.f;          // lazy-rescale threshold (log2 units)

typedef __attribute__((address_space(3))) void lds_void;

__device__ inline int swz(int row) { return ((row & 3) << 2) ^ ((row >> 2) & 3); }

__device__ inline uint32_t cvt2(float a, float b) {
    bf16x2 v;
    v[0] = static_cast<__bf16>(a);
    v[1] = static_cast<__bf16>(b);
    return __builtin_bit_cast(uint32_t, v);
}

__device__ inline float dot2_ones(uint32_t p, float acc) {
    const bf16x2 one = {static_cast<__bf16>(1.f), static_cast<__bf16>(1.f)};
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, p), one, acc, false);
}

// Transposing LDS read: within each 16-lane group, lane s points at 4
// consecutive elements of a row; lane 4a+b receives element b of the chunks of
// lanes a, a+4, a+8, a+12.
__device__ inline i16x4 lds_read_tr(const char *p) {
    return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        reinterpret_cast<__attribute__((address_space(3))) i16x4 *>(reinterpret_cast<uintptr_t>(p)));
}

__global__ void __launch_bounds__(kThreads, 1)
k_prefill_attn(const uint16_t *__restrict__ kpool, const uint16_t *__restrict__ vpool,
               const uint16_t *__restrict__ q, uint16_t *__restrict__ out,
               const int32_t *__restrict__ qo_indptr, const int32_t *__restrict__ prefix_lens,
               const int32_t *__restrict__ bt, int bt_stride, int hkv, int group, int num_pages,
               float scale_log2, int max_qblocks, int n_hgroups) {
    __shared__ __attribute__((aligned(1024))) uint16_t s_k[2 * TILE];
    __shared__ __attribute__((aligned(1024))) uint16_t s_v[2 * TILE];
    __shared__ int32_t s_bt[kBtCache];

    const int b = blockIdx.y;
    const int x = blockIdx.x;
    const int kvh = x % hkv;
    const int hg = (x / hkv) % n_hgroups;
    const int qblk = max_qblocks - 1 - x / (hkv * n_hgroups);  // heaviest blocks first
    const int row0 = qo_indptr[b];
    const int n = qo_indptr[b + 1] - row0;
    if (qblk * BM >= n) return;
    const int r = prefix_lens[b];
    const int32_t *btrow = bt + static_cast<size_t>(b) * bt_stride;
    const int np_seq = min((r + n + kPageSize - 1) / kPageSize, bt_stride);
    const int kv_end = r + min(qblk * BM + BM, n);
    const int nt = (kv_end + BN - 1) / BN;

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // uniform per wave
    const int hl = hg * 4 + (wave & 3);  // head within the kv group
    const bool active = hl < group;
    const int hq = hkv * group;
    const int h = kvh * group + (active ? hl : 0);
    const int l32 = lane & 31, g = lane >> 5;
    const int pos = qblk * BM + (wave >> 2) * 32 + l32;  // this lane's query column
    const int qabs = r + pos;
    const int diag = r + qblk * BM + (wave >> 2) * 32;  // smallest query of the wave

    // block-table entries of this work-group's keys
    const int np_wg = min(4 * nt, np_seq);
    for (int i = threadIdx.x; i < min(np_wg, kBtCache); i += kThreads) s_bt[i] = btrow[i];
    const int first_page = btrow[0];
    const int safe_page = (first_page >= 0 && first_page < num_pages) ? first_page : 0;

    // Q^T operand, all 8 dim-steps (k = 16*kb + 8*g + e)
    uint4 qop[8];
    {
        const bool ok = active && pos < n;
        const uint16_t *qp = q + (static_cast<size_t>(row0 + (ok ? pos : 0)) * hq + h) * kHeadDim + 8 * g;
#pragma unroll
        for (int kb = 0; kb < 8; ++kb)
            qop[kb] = ok ? *reinterpret_cast<const uint4 *>(qp + 16 * kb) : make_uint4(0, 0, 0, 0);
    }

    // ---- per-lane byte offsets, computed once
    // K operand: row l32 (+32 rows for the second key block), logical chunk 2kb+g
    int koff[8];
#pragma unroll
    for (int kb = 0; kb < 8; ++kb) koff[kb] = l32 * 256 + 16 * ((2 * kb + g) ^ swz(l32));
    // V transposing reads: lane s of 16-lane group q reads row 8hh + 4(q/2) + s/4
    // (+16 ks) at dims 32db + 16(q%2) + 4(s%4): logical chunk 4db + 2(q%2) + (s%4)/2
    int voff[2][4];
    {
        const int q16 = lane >> 4, s16 = lane & 15;
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
            const int row = 8 * hh + 4 * (q16 >> 1) + (s16 >> 2);
#pragma unroll
            for (int db = 0; db < 4; ++db) {
                const int chunk = (4 * db + 2 * (q16 & 1) + ((s16 & 3) >> 1)) ^ swz(row);
                voff[hh][db] = row * 256 + 16 * chunk + 8 * (s16 & 1);
            }
        }
    }
    // direct loads: wave w moves rows 8w + 4j + lane/16 of a tile (j = 0, 1), all
    // in page w/2 of the tile; lane i lands in physical chunk i%16
    int goff[2];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
        const int row = 8 * wave + 4 * j + (lane >> 4);
        goff[j] = (row & 15) * kHeadDim + 8 * ((lane & 15) ^ swz(row));
    }

    f32x16 oacc[4];
#pragma unroll
    for (int db = 0; db < 4; ++db)
#pragma unroll
        for (int i = 0; i < 16; ++i) oacc[db][i] = 0.f;
    float m_run = -INFINITY;
    float l_run = 0.f;

    __syncthreads();  // s_bt

    // Issues the direct loads of tile `it` into buffer `buf`.
    auto tile_dma = [&](int it, int buf) {
        const int p = 4 * it + (wave >> 1);  // uniform: this wave's page of the tile
        int page;
        if (p < np_seq) {
            page = p < kBtCache ? __builtin_amdgcn_readfirstlane(s_bt[p]) : btrow[p];
            // a page outside the pool is never read (see below)
            if (page < 0 || page >= num_pages) page = safe_page;
        } else {
            // a page past the sequence is read from the sequence's first page:
            // those keys lie past every valid query and the causal mask discards
            // them, and that page holds finite data
            page = safe_page;
        }
        const uint16_t *kp = kpool + (static_cast<size_t>(page) * hkv + kvh) * (kPageSize * kHeadDim);
        const uint16_t *vp = vpool + (static_cast<size_t>(page) * hkv + kvh) * (kPageSize * kHeadDim);
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int lrow = 8 * wave + 4 * j;
            __builtin_amdgcn_global_load_lds(kp + goff[j],
                                             reinterpret_cast<lds_void *>(reinterpret_cast<uintptr_t>(
                                                 s_k + buf * TILE + lrow * ROW)),
                                             16, 0, 0);
            __builtin_amdgcn_global_load_lds(vp + goff[j],
                                             reinterpret_cast<lds_void *>(reinterpret_cast<uintptr_t>(
                                                 s_v + buf * TILE + lrow * ROW)),
                                             16, 0, 0);
        }
    };

    auto tile_compute = [&](int it, int buf) {
        const char *kb_ = reinterpret_cast<const char *>(s_k + buf * TILE);
        const char *vb_ = reinterpret_cast<const char *>(s_v + buf * TILE);
        // ---- S^T = K Q^T : two 32-key blocks
        f32x16 sacc[2];
#pragma unroll
        for (int blk = 0; blk < 2; ++blk)
#pragma unroll
            for (int i = 0; i < 16; ++i) sacc[blk][i] = 0.f;
#pragma unroll
        for (int kb = 0; kb < 8; ++kb)
#pragma unroll
            for (int blk = 0; blk < 2; ++blk) {
                const bf16x8 a = *reinterpret_cast<const bf16x8 *>(kb_ + blk * 32 * 256 + koff[kb]);
                sacc[blk] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, __builtin_bit_cast(bf16x8, qop[kb]),
                                                                    sacc[blk], 0, 0, 0);
            }
        // ---- causal mask on tiles crossing the diagonal
        const int k0 = it * BN;
        if (k0 + BN - 1 > diag) {
#pragma unroll
            for (int blk = 0; blk < 2; ++blk)
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const int key = k0 + 32 * blk + 8 * (i >> 2) + 4 * g + (i & 3);
                    if (key > qabs) sacc[blk][i] = -INFINITY;
                }
        }
        // ---- online softmax (base 2)
        float mx = -INFINITY;
#pragma unroll
        for (int blk = 0; blk < 2; ++blk)
#pragma unroll
            for (int i = 0; i < 16; ++i) mx = fmaxf(mx, sacc[blk][i]);
        mx = fmaxf(mx, __shfl_xor(mx, 32));  // lanes l and l^32 hold the same query
        const float m_tile = mx * scale_log2;
        if (__builtin_amdgcn_ballot_w64(m_tile > m_run + kRescaleLog2) != 0) {
            const float m_new = fmaxf(m_run, m_tile);
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
        uint4 pop[4];
#pragma unroll
        for (int kstep = 0; kstep < 4; ++kstep) {
            const int blk = kstep >> 1, a8 = (kstep & 1) * 8;
            float p[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) p[e] = __builtin_amdgcn_exp2f(fmaf(sacc[blk][a8 + e], scale_log2, -m_run));
            pop[kstep] = make_uint4(cvt2(p[0], p[1]), cvt2(p[2], p[3]), cvt2(p[4], p[5]), cvt2(p[6], p[7]));
            l_run = dot2_ones(pop[kstep].x, l_run);
            l_run = dot2_ones(pop[kstep].y, l_run);
            l_run = dot2_ones(pop[kstep].z, l_run);
            l_run = dot2_ones(pop[kstep].w, l_run);
        }
        // ---- O^T += V^T P^T ; V^T operand = two transposing reads (e = 0..3, 4..7)
#pragma unroll
        for (int kstep = 0; kstep < 4; ++kstep)
#pragma unroll
            for (int db = 0; db < 4; ++db) {
                const i16x4 lo = lds_read_tr(vb_ + kstep * 16 * 256 + voff[0][db]);
                const i16x4 hi = lds_read_tr(vb_ + kstep * 16 * 256 + voff[1][db]);
                const bf16x8 a = __builtin_bit_cast(
                    bf16x8, make_uint4(__builtin_bit_cast(uint2, lo).x, __builtin_bit_cast(uint2, lo).y,
                                       __builtin_bit_cast(uint2, hi).x, __builtin_bit_cast(uint2, hi).y));
                oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, __builtin_bit_cast(bf16x8, pop[kstep]),
                                                                   oacc[db], 0, 0, 0);
            }
    };

    auto step = [&](int it, int buf) {
        const bool more = it + 1 < nt;
        if (more) tile_dma(it + 1, buf ^ 1);
        if (active) tile_compute(it, buf);
        if (more) __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): this wave's direct loads landed
        __syncthreads();
    };

    tile_dma(0, 0);
    __builtin_amdgcn_s_waitcnt(0x0F70);
    __syncthreads();
    for (int it = 0; it < nt; it += 2) {  // unrolled by the buffer parity
        step(it, 0);
        if (it + 1 < nt) step(it + 1, 1);
    }

    // ---- normalise and write O[pos][h][d] (4 consecutive dims per store)
    const float lt = l_run + __shfl_xor(l_run, 32);
    if (!active || pos >= n) return;
    const float inv = 1.f / lt;
    uint16_t *op = out + (static_cast<size_t>(row0 + pos) * hq + h) * kHeadDim;
#pragma unroll
    for (int db = 0; db < 4; ++db)
#pragma unroll
        for (int i4 = 0; i4 < 4; ++i4) {
            const int d0 = 32 * db + 8 * i4 + 4 * g;
            *reinterpret_cast<uint2 *>(op + d0) =
                make_uint2(cvt2(oacc[db][4 * i4 + 0] * inv, oacc[db][4 * i4 + 1] * inv),
                           cvt2(oacc[db][4 * i4 + 2] * inv, oacc[db][4 * i4 + 3] * inv));
        }
}

}  // namespace

extern "C" mw_status mw_prefill_attn(const mw_kv_pool *pool, const mw_attn_shape *shape, int32_t batch,
                                     const int32_t *h_new_lens, const int32_t *h_prefix_lens,
                                     const int32_t *d_qo_indptr, const int32_t *d_prefix_lens,
                                     const int32_t *d_block_table, int32_t bt_stride, const void *d_q,
                                     void *d_out, mw_stream stream, mw_timing *timing) {
    const char *who = "mw_prefill_attn";
    if (!pool || !shape || batch < 0 || batch > 65535 || bt_stride < 1 ||
        (batch > 0 && (!h_new_lens || !h_prefix_lens)))
        return fail(MW_ERR_INVALID_ARG, "%s: bad arguments", who);
    if (shape->head_dim != kHeadDim) return fail(MW_ERR_UNSUPPORTED, "%s: head_dim must be 128", who);
    if (!(shape->scale > 0.f) || !(shape->scale < INFINITY))
        return fail(MW_ERR_INVALID_ARG, "%s: scale must be positive and finite", who);
    if (shape->num_kv_heads != pool->desc.num_kv_heads || shape->num_q_heads < 1 ||
        shape->num_q_heads % shape->num_kv_heads)
        return fail(MW_ERR_INVALID_ARG, "%s: num_q_heads must be a multiple of the pool's %d kv heads", who,
                    pool->desc.num_kv_heads);
    int64_t max_n = 0;
    for (int32_t b = 0; b < batch; ++b) {
        if (h_new_lens[b] < 0 || h_prefix_lens[b] < 0 ||
            static_cast<int64_t>(h_new_lens[b]) + h_prefix_lens[b] > static_cast<int64_t>(bt_stride) * kPageSize)
            return fail(MW_ERR_INVALID_ARG, "%s: sequence %d: prefix %d + new %d exceeds %d table pages", who, b,
                        h_prefix_lens[b], h_new_lens[b], bt_stride);
        max_n = h_new_lens[b] > max_n ? h_new_lens[b] : max_n;
    }
    if (max_n > 0 && (!d_qo_indptr || !d_prefix_lens || !d_block_table || !d_q || !d_out))
        return fail(MW_ERR_INVALID_ARG, "%s: NULL device pointer", who);
    if (max_n > 0 && (!aligned16(d_q) || !aligned16(d_out)))
        return fail(MW_ERR_INVALID_ARG, "%s: Q and O must be 16-byte aligned", who);
    hipStream_t s = static_cast<hipStream_t>(stream);
    mw_status st = timing_begin(timing, s);
    if (st != MW_OK) return st;
    if (max_n > 0) {
        const int hkv = shape->num_kv_heads;
        const int group = shape->num_q_heads / hkv;
        const int n_hgroups = (group + 3) / 4;
        const int64_t max_qblocks = (max_n + BM - 1) / BM;
        const int64_t gx = max_qblocks * hkv * n_hgroups;
        if (gx > 0x7fffffff) return fail(MW_ERR_UNSUPPORTED, "%s: grid too large", who);
        hipLaunchKernelGGL(k_prefill_attn, dim3(static_cast<unsigned>(gx), batch), dim3(kThreads), 0, s, pool->k,
                           pool->v, static_cast<const uint16_t *>(d_q), static_cast<uint16_t *>(d_out), d_qo_indptr,
                           d_prefix_lens, d_block_table, bt_stride, hkv, group, pool->desc.num_pages,
                           shape->scale * kLog2e, static_cast<int>(max_qblocks), n_hgroups);
        st = check_launch("k_prefill_attn");
        if (st != MW_OK) return st;
    }
    st = timing_kernel_done(timing, s);
    timing_end(timing);
    return st;
}
