// Causal prefill attention of a chunk of new tokens over its cached prefix.
//
// Prefill is compute-bound (paper Sec. 2.2; Sec. 3.3, Table
// "tab:theory_cost": O(n d^2 + L n d) with L = r + n), so both contractions
// run on the bf16 matrix cores (fp32 accumulate) and the loop is organised
// around MFMA throughput.
//
// Work-group = 8 waves = 64 query positions x 4 query heads of one kv head;
// wave w owns head (w % 4) of the group and positions 32*(w / 4) .. +31, so
// every K/V tile staged in LDS serves 4 heads x 64 positions.  Two waves share
// each SIMD: while one runs its softmax on the vector ALU the other keeps the
// matrix core busy, and each wave's state (Q^T, S, O, P: about 150 registers)
// stays in ordinary VGPRs.
// Key tiles of 64 keys = 4 pages are copied into LDS row-major, double-buffered:
//   K tile [64 keys][128 dims]  row stride 136 (16-byte operand reads are
//                               bank-conflict free)
//   V tile [64 keys][128 dims]  row stride 160 (conflict-free transposing reads)
// Per tile and wave:
//   S^T[key][q] = K Q^T      32x32x16 MFMA; A = K rows from LDS, B = Q^T held in
//                            registers for the whole kernel
//   online softmax in base 2 (scores scaled by scale*log2 e inside one FMA);
//   the causal mask is applied only on tiles that cross the diagonal
//   O^T[d][q] += V^T P^T     32x32x16 MFMA; A = V^T gathered by the LDS
//                            transposing read (ds_read_b64_tr_b16), B = P^T taken
//                            straight from the S^T accumulators as bf16
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
constexpr int KSTR = 136;                    // K tile row stride (bf16 elements)
constexpr int VSTR = 160;                    // V tile row stride (bf16 elements)
constexpr int K_ELEMS = BN * KSTR;
constexpr int V_ELEMS = BN * VSTR;
constexpr int STAGE = K_ELEMS + V_ELEMS;     // one buffer, bf16 elements
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kRescaleLog2 = 8.f;          // lazy-rescale threshold (log2 units)

__device__ inline uint32_t cvt2(float a, float b) {
    bf16x2 v;
    v[0] = static_cast<__bf16>(a);
    v[1] = static_cast<__bf16>(b);
    return __builtin_bit_cast(uint32_t, v);
}

__device__ inline uint4 sel4(bool ok, uint4 v) {
    return make_uint4(ok ? v.x : 0u, ok ? v.y : 0u, ok ? v.z : 0u, ok ? v.w : 0u);
}

// Transposing LDS read: within each 16-lane group, lane s points at 4
// consecutive elements of a row; lane 4a+b receives element b of the chunks of
// lanes a, a+4, a+8, a+12.
__device__ inline i16x4 lds_read_tr(const uint16_t *p) {
    return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        reinterpret_cast<__attribute__((address_space(3))) i16x4 *>(
            reinterpret_cast<uintptr_t>(p)));
}

struct TileRegs {
    uint4 k[2];
    uint4 v[2];
    bool ok[2];
};

// Global -> registers for key tile `it`: thread t copies 16-byte chunk t%16 of
// keys t/16 and t/16 + 32 for both K and V.  Pages past the sequence (or with
// an index outside the pool) read page 0 and are zeroed at the store, so no
// branch separates the loads from the compute that follows.
__device__ inline void tile_load(TileRegs &tr, const uint16_t *__restrict__ kpool,
                                 const uint16_t *__restrict__ vpool, const int32_t *__restrict__ btrow,
                                 int it, int np_seq, int hkv, int kvh, int num_pages) {
    const int t = threadIdx.x;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
        const int key = (t >> 4) + 32 * j;
        const int p = 4 * it + (key >> 4);
        const int page = btrow[p < np_seq ? p : 0];
        tr.ok[j] = p < np_seq && page >= 0 && page < num_pages;
        const size_t off = ((static_cast<size_t>(tr.ok[j] ? page : 0) * hkv + kvh) * kPageSize + (key & 15)) *
                               kHeadDim + 8 * (t & 15);
        tr.k[j] = *reinterpret_cast<const uint4 *>(kpool + off);
        tr.v[j] = *reinterpret_cast<const uint4 *>(vpool + off);
    }
}

__device__ inline void tile_store(const TileRegs &tr, uint16_t *stage) {
    const int t = threadIdx.x;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
        const int key = (t >> 4) + 32 * j;
        *reinterpret_cast<uint4 *>(stage + key * KSTR + 8 * (t & 15)) = sel4(tr.ok[j], tr.k[j]);
        *reinterpret_cast<uint4 *>(stage + K_ELEMS + key * VSTR + 8 * (t & 15)) = sel4(tr.ok[j], tr.v[j]);
    }
}

__global__ void __launch_bounds__(kThreads, 1)
k_prefill_attn(const uint16_t *__restrict__ kpool, const uint16_t *__restrict__ vpool,
               const uint16_t *__restrict__ q, uint16_t *__restrict__ out,
               const int32_t *__restrict__ qo_indptr, const int32_t *__restrict__ prefix_lens,
               const int32_t *__restrict__ bt, int bt_stride, int hkv, int group, int num_pages,
               float scale_log2, int max_qblocks, int n_hgroups) {
    __shared__ __attribute__((aligned(16))) uint16_t lds[2 * STAGE];

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

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int hl = hg * 4 + (wave & 3);  // head within the kv group
    const bool active = hl < group;
    const int hq = hkv * group;
    const int h = kvh * group + (active ? hl : 0);
    const int l32 = lane & 31, g = lane >> 5;
    const int pos = qblk * BM + (wave >> 2) * 32 + l32;  // this lane's query column
    const int qabs = r + pos;
    const int diag = r + qblk * BM + (wave >> 2) * 32;  // smallest query of the wave

    // Q^T operand, all 8 dim-steps (k = 16*kb + 8*g + e)
    uint4 qop[8];
    {
        const bool ok = active && pos < n;
        const uint16_t *qp = q + (static_cast<size_t>(row0 + (ok ? pos : 0)) * hq + h) * kHeadDim + 8 * g;
#pragma unroll
        for (int kb = 0; kb < 8; ++kb)
            qop[kb] = ok ? *reinterpret_cast<const uint4 *>(qp + 16 * kb) : make_uint4(0, 0, 0, 0);
    }

    f32x16 oacc[4];
#pragma unroll
    for (int db = 0; db < 4; ++db)
#pragma unroll
        for (int i = 0; i < 16; ++i) oacc[db][i] = 0.f;
    float m_run = -INFINITY;
    float l_run = 0.f;

    // transposing-read addresses inside a V tile (see lds_read_tr): lane s of
    // group q reads key 8h + 4(q/2) + s/4 (+16 ks), dims 16(q%2) + 4(s%4) (+32 db)
    const int grp16 = lane >> 4, s16 = lane & 15;
    const int vtr_off = (4 * (grp16 >> 1) + (s16 >> 2)) * VSTR + 16 * (grp16 & 1) + 4 * (s16 & 3);

    TileRegs tr;
    tile_load(tr, kpool, vpool, btrow, 0, np_seq, hkv, kvh, num_pages);
    tile_store(tr, lds);
    __syncthreads();

    for (int it = 0; it < nt; ++it) {
        const bool more = it + 1 < nt;
        if (more) tile_load(tr, kpool, vpool, btrow, it + 1, np_seq, hkv, kvh, num_pages);
        const uint16_t *ks = lds + (it & 1) * STAGE;
        const uint16_t *vs = ks + K_ELEMS;
        if (active) {
            // ---- S^T = K Q^T : two 32-key blocks
            f32x16 sacc[2];
#pragma unroll
            for (int kblk = 0; kblk < 2; ++kblk)
#pragma unroll
                for (int i = 0; i < 16; ++i) sacc[kblk][i] = 0.f;
#pragma unroll
            for (int kb = 0; kb < 8; ++kb)
#pragma unroll
                for (int kblk = 0; kblk < 2; ++kblk) {
                    const bf16x8 a = *reinterpret_cast<const bf16x8 *>(ks + (32 * kblk + l32) * KSTR + 16 * kb + 8 * g);
                    sacc[kblk] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, __builtin_bit_cast(bf16x8, qop[kb]),
                                                                         sacc[kblk], 0, 0, 0);
                }
            // ---- causal mask on tiles crossing the diagonal
            const int k0 = it * BN;
            if (k0 + BN - 1 > diag) {
#pragma unroll
                for (int kblk = 0; kblk < 2; ++kblk)
#pragma unroll
                    for (int i = 0; i < 16; ++i) {
                        const int key = k0 + 32 * kblk + 8 * (i >> 2) + 4 * g + (i & 3);
                        if (key > qabs) sacc[kblk][i] = -INFINITY;
                    }
            }
            // ---- online softmax (base 2)
            float mx = -INFINITY;
#pragma unroll
            for (int kblk = 0; kblk < 2; ++kblk)
#pragma unroll
                for (int i = 0; i < 16; ++i) mx = fmaxf(mx, sacc[kblk][i]);
            mx = fmaxf(mx, __shfl_xor(mx, 32));
            // The reference maximum m_run moves only when a column's maximum
            // exceeds it by more than 2^8: every exp2 below then stays <= 256 and
            // O, l need no rescaling on most tiles.  O / l does not depend on the
            // reference used.
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
            float p[2][16];
            float ls = 0.f;
#pragma unroll
            for (int kblk = 0; kblk < 2; ++kblk)
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    p[kblk][i] = __builtin_amdgcn_exp2f(fmaf(sacc[kblk][i], scale_log2, -m_run));
                    ls += p[kblk][i];
                }
            l_run += ls;
            // key-step ks covers keys 16ks..16ks+15 = registers 8a..8a+7 of block ks/2
            uint4 pop[4];
#pragma unroll
            for (int kstep = 0; kstep < 4; ++kstep) {
                const int kblk = kstep >> 1, a8 = (kstep & 1) * 8;
                pop[kstep] = make_uint4(cvt2(p[kblk][a8 + 0], p[kblk][a8 + 1]), cvt2(p[kblk][a8 + 2], p[kblk][a8 + 3]),
                                        cvt2(p[kblk][a8 + 4], p[kblk][a8 + 5]), cvt2(p[kblk][a8 + 6], p[kblk][a8 + 7]));
            }
            // ---- O^T += V^T P^T ; V^T operand = two transposing reads (e = 0..3, 4..7)
#pragma unroll
            for (int kstep = 0; kstep < 4; ++kstep)
#pragma unroll
                for (int db = 0; db < 4; ++db) {
                    const uint16_t *vp = vs + vtr_off + 16 * kstep * VSTR + 32 * db;
                    const i16x4 lo = lds_read_tr(vp);
                    const i16x4 hi = lds_read_tr(vp + 8 * VSTR);
                    const bf16x8 a = __builtin_bit_cast(
                        bf16x8, make_uint4(__builtin_bit_cast(uint2, lo).x, __builtin_bit_cast(uint2, lo).y,
                                           __builtin_bit_cast(uint2, hi).x, __builtin_bit_cast(uint2, hi).y));
                    oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, __builtin_bit_cast(bf16x8, pop[kstep]),
                                                                       oacc[db], 0, 0, 0);
                }
        }
        if (more) tile_store(tr, lds + ((it + 1) & 1) * STAGE);
        __syncthreads();
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
