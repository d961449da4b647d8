// Causal prefill attention of a chunk of new tokens over its cached prefix.
//
// Prefill is compute-bound (paper Sec. 2.2; Sec. 3.3, Table
// "tab:theory_cost": O(n d^2 + L n d) with L = r + n), so both contractions
// run on the bf16 matrix cores (fp32 accumulate) and the loop is organised
// around MFMA throughput.
//
// Work-group = 4 waves = 64 query positions x 4 query heads of one kv head;
// each wave owns one head and all 64 positions (two 32-column MFMA blocks),
// so every K/V tile staged in LDS serves 4 heads x 64 positions.
// Key tiles of 64 keys = 4 pages are staged through LDS, double-buffered:
//   K  tile [64 keys][128 dims]   (row stride 136: conflict-free 16-B reads)
//   V^T tile [128 dims][64 keys]  (row stride 72), transposed on the way in
//       and with key bits 2 and 3 swapped inside each 16-key group, so that
//       one 16-byte read yields exactly the keys that the probability
//       operand holds (see pv_key below).
// Per tile and wave:
//   S^T[key][q] = K Q^T      32x32x16 MFMA, A = K rows from LDS, B = Q^T held
//                            in registers for the whole kernel
//   online softmax in base 2 (scores scaled by scale*log2 e inside one FMA),
//   causal mask only on tiles that cross the diagonal
//   O^T[d][q] += V^T P^T     32x32x16 MFMA, B = P^T taken straight from the
//                            S^T accumulators (converted to bf16)
// Causal position: query row i of a sequence with prefix r sees keys
// 0 .. r + i (bottom-right alignment; a chunk reads every earlier chunk's KV).
#include "mw_internal.h"

using namespace mw;

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kThreads = 256;
constexpr int BM = 64;                       // query positions per work-group
constexpr int BN = 64;                       // keys per tile
constexpr int KSTR = 136;                    // K tile row stride (bf16 elements)
constexpr int VSTR = 72;                     // V^T tile row stride (bf16 elements)
constexpr int K_ELEMS = BN * KSTR;
constexpr int V_ELEMS = kHeadDim * VSTR;
constexpr int STAGE = K_ELEMS + V_ELEMS;     // one buffer, bf16 elements
constexpr float kLog2e = 1.4426950408889634f;

__device__ inline uint32_t pack_lo(uint32_t a, uint32_t b) { return (a & 0xffffu) | (b << 16); }
__device__ inline uint32_t pack_hi(uint32_t a, uint32_t b) { return (a >> 16) | (b & 0xffff0000u); }

// Column of key k (0..63) inside the V^T tile: bits 2 and 3 swapped.
__device__ inline int pv_col(int k) { return (k & ~12) | ((k & 4) << 1) | ((k & 8) >> 1); }

__device__ inline uint32_t cvt2(float a, float b) {
    bf16x2 v;
    v[0] = static_cast<__bf16>(a);
    v[1] = static_cast<__bf16>(b);
    return __builtin_bit_cast(uint32_t, v);
}

struct TileRegs {
    uint4 k[4];
    uint4 v[4];
};

// Global -> registers for key tile `it`.  Pages past the sequence (or with an
// index outside the pool) are read as zeros.
__device__ inline void tile_load(TileRegs &tr, const uint16_t *__restrict__ kpool,
                                 const uint16_t *__restrict__ vpool, const int32_t *__restrict__ btrow,
                                 int it, int np_seq, int hkv, int kvh, int num_pages) {
    const int t = threadIdx.x;
    const uint4 z = make_uint4(0, 0, 0, 0);
    // K: load j reads page j of the tile, slot t/16, 16-byte chunk t%16
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int p = 4 * it + j;
        const int page = p < np_seq ? btrow[p] : -1;
        const bool ok = page >= 0 && page < num_pages;
        const size_t off = ((static_cast<size_t>(ok ? page : 0) * hkv + kvh) * kPageSize + (t >> 4)) * kHeadDim +
                           8 * (t & 15);
        tr.k[j] = ok ? *reinterpret_cast<const uint4 *>(kpool + off) : z;
    }
    // V: thread owns keys 4*(t/16)+kk (kk = 0..3) and dims 8*(t%16)..+7
    {
        const int key4 = t >> 4;
        const int p = 4 * it + (key4 >> 2);
        const int page = p < np_seq ? btrow[p] : -1;
        const bool ok = page >= 0 && page < num_pages;
        const size_t base =
            ((static_cast<size_t>(ok ? page : 0) * hkv + kvh) * kPageSize + 4 * (key4 & 3)) * kHeadDim + 8 * (t & 15);
#pragma unroll
        for (int kk = 0; kk < 4; ++kk)
            tr.v[kk] = ok ? *reinterpret_cast<const uint4 *>(vpool + base + kk * kHeadDim) : z;
    }
}

// Registers -> LDS stage (K rows as loaded; V transposed with permuted keys).
__device__ inline void tile_store(const TileRegs &tr, uint16_t *stage) {
    const int t = threadIdx.x;
    uint16_t *ks = stage;
    uint16_t *vs = stage + K_ELEMS;
#pragma unroll
    for (int j = 0; j < 4; ++j)
        *reinterpret_cast<uint4 *>(ks + (16 * j + (t >> 4)) * KSTR + 8 * (t & 15)) = tr.k[j];
    const int key0 = 4 * (t >> 4);
    const int col = pv_col(key0);
    const int d0 = 8 * (t & 15);
    const uint32_t *w0 = reinterpret_cast<const uint32_t *>(&tr.v[0]);
    const uint32_t *w1 = reinterpret_cast<const uint32_t *>(&tr.v[1]);
    const uint32_t *w2 = reinterpret_cast<const uint32_t *>(&tr.v[2]);
    const uint32_t *w3 = reinterpret_cast<const uint32_t *>(&tr.v[3]);
#pragma unroll
    for (int m = 0; m < 4; ++m) {
        // dims d0+2m (low halves) and d0+2m+1 (high halves) of the 4 keys
        *reinterpret_cast<uint2 *>(vs + (d0 + 2 * m) * VSTR + col) =
            make_uint2(pack_lo(w0[m], w1[m]), pack_lo(w2[m], w3[m]));
        *reinterpret_cast<uint2 *>(vs + (d0 + 2 * m + 1) * VSTR + col) =
            make_uint2(pack_hi(w0[m], w1[m]), pack_hi(w2[m], w3[m]));
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
    const int diag = r + qblk * BM;  // smallest absolute query position of the block

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int hl = hg * 4 + wave;  // head within the kv group
    const bool active = hl < group;
    const int hq = hkv * group;
    const int h = kvh * group + (active ? hl : 0);
    const int l32 = lane & 31, g = lane >> 5;

    // Q^T operand for both 32-position blocks, all 8 dim-steps
    uint4 qop[2][8];
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
        const int pos = qblk * BM + qb * 32 + l32;
        const bool ok = active && pos < n;
        const uint16_t *qp = q + (static_cast<size_t>(row0 + (ok ? pos : 0)) * hq + h) * kHeadDim + 8 * g;
#pragma unroll
        for (int kb = 0; kb < 8; ++kb)
            qop[qb][kb] = ok ? *reinterpret_cast<const uint4 *>(qp + 16 * kb) : make_uint4(0, 0, 0, 0);
    }

    f32x16 oacc[4][2];
#pragma unroll
    for (int db = 0; db < 4; ++db)
#pragma unroll
        for (int qb = 0; qb < 2; ++qb)
#pragma unroll
            for (int i = 0; i < 16; ++i) oacc[db][qb][i] = 0.f;
    float m_run[2] = {-INFINITY, -INFINITY};
    float l_run[2] = {0.f, 0.f};

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
            // ---- S^T = K Q^T
            f32x16 sacc[2][2];
#pragma unroll
            for (int kblk = 0; kblk < 2; ++kblk)
#pragma unroll
                for (int qb = 0; qb < 2; ++qb)
#pragma unroll
                    for (int i = 0; i < 16; ++i) sacc[kblk][qb][i] = 0.f;
#pragma unroll
            for (int kb = 0; kb < 8; ++kb) {
#pragma unroll
                for (int kblk = 0; kblk < 2; ++kblk) {
                    const bf16x8 a = *reinterpret_cast<const bf16x8 *>(ks + (32 * kblk + l32) * KSTR + 16 * kb + 8 * g);
#pragma unroll
                    for (int qb = 0; qb < 2; ++qb)
                        sacc[kblk][qb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                            a, __builtin_bit_cast(bf16x8, qop[qb][kb]), sacc[kblk][qb], 0, 0, 0);
                }
            }
            // ---- causal mask on tiles crossing the diagonal
            const int k0 = it * BN;
            if (k0 + BN - 1 > diag) {
#pragma unroll
                for (int qb = 0; qb < 2; ++qb) {
                    const int qabs = r + qblk * BM + qb * 32 + l32;
#pragma unroll
                    for (int kblk = 0; kblk < 2; ++kblk)
#pragma unroll
                        for (int i = 0; i < 16; ++i) {
                            const int key = k0 + 32 * kblk + 8 * (i >> 2) + 4 * g + (i & 3);
                            if (key > qabs) sacc[kblk][qb][i] = -INFINITY;
                        }
                }
            }
            // ---- online softmax (base 2) and P^T operands
            uint4 pop[2][4];
#pragma unroll
            for (int qb = 0; qb < 2; ++qb) {
                float mx = -INFINITY;
#pragma unroll
                for (int kblk = 0; kblk < 2; ++kblk)
#pragma unroll
                    for (int i = 0; i < 16; ++i) mx = fmaxf(mx, sacc[kblk][qb][i]);
                mx = fmaxf(mx, __shfl_xor(mx, 32));
                const float m_new = fmaxf(m_run[qb], mx * scale_log2);
                const float alpha = __builtin_amdgcn_exp2f(m_run[qb] - m_new);
                m_run[qb] = m_new;
                float ls = 0.f;
                float p[2][16];
#pragma unroll
                for (int kblk = 0; kblk < 2; ++kblk)
#pragma unroll
                    for (int i = 0; i < 16; ++i) {
                        p[kblk][i] = __builtin_amdgcn_exp2f(fmaf(sacc[kblk][qb][i], scale_log2, -m_new));
                        ls += p[kblk][i];
                    }
                l_run[qb] = l_run[qb] * alpha + ls;
#pragma unroll
                for (int db = 0; db < 4; ++db)
#pragma unroll
                    for (int i = 0; i < 16; ++i) oacc[db][qb][i] *= alpha;
                // key-step ks covers keys 16ks..16ks+15 = registers 8a..8a+7 of block ks/2
#pragma unroll
                for (int ks = 0; ks < 4; ++ks) {
                    const int kblk = ks >> 1, a8 = (ks & 1) * 8;
                    pop[qb][ks] = make_uint4(cvt2(p[kblk][a8 + 0], p[kblk][a8 + 1]), cvt2(p[kblk][a8 + 2], p[kblk][a8 + 3]),
                                             cvt2(p[kblk][a8 + 4], p[kblk][a8 + 5]), cvt2(p[kblk][a8 + 6], p[kblk][a8 + 7]));
                }
            }
            // ---- O^T += V^T P^T
#pragma unroll
            for (int ks = 0; ks < 4; ++ks) {
#pragma unroll
                for (int db = 0; db < 4; ++db) {
                    const bf16x8 a = *reinterpret_cast<const bf16x8 *>(vs + (32 * db + l32) * VSTR + 16 * ks + 8 * g);
#pragma unroll
                    for (int qb = 0; qb < 2; ++qb)
                        oacc[db][qb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                            a, __builtin_bit_cast(bf16x8, pop[qb][ks]), oacc[db][qb], 0, 0, 0);
                }
            }
        }
        if (more) tile_store(tr, lds + ((it + 1) & 1) * STAGE);
        __syncthreads();
    }

    if (!active) return;
    // ---- normalise and write O[pos][h][d] (4 consecutive dims per store)
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
        const float lt = l_run[qb] + __shfl_xor(l_run[qb], 32);
        const float inv = 1.f / lt;
        const int pos = qblk * BM + qb * 32 + l32;
        if (pos >= n) continue;
        uint16_t *op = out + (static_cast<size_t>(row0 + pos) * hq + h) * kHeadDim;
#pragma unroll
        for (int db = 0; db < 4; ++db)
#pragma unroll
            for (int i4 = 0; i4 < 4; ++i4) {
                const int d0 = 32 * db + 8 * i4 + 4 * g;
                const f32x16 &o = oacc[db][qb];
                *reinterpret_cast<uint2 *>(op + d0) =
                    make_uint2(cvt2(o[4 * i4 + 0] * inv, o[4 * i4 + 1] * inv),
                               cvt2(o[4 * i4 + 2] * inv, o[4 * i4 + 3] * inv));
            }
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
