// Causal prefill attention of a chunk of new tokens over its cached prefix:
// the kernel (its work-group body is in prefill_block.h) and its launch.
#include <algorithm>
#include <vector>

#include "prefill_block.h"

using namespace mw;

namespace {

using namespace pf;

template <bool kTableInLds, int NW>
__global__ void __launch_bounds__(64 * NW, NW == 4 ? 2 : 1)
k_prefill_attn(const uint16_t *__restrict__ kpool, const uint16_t *__restrict__ vpool,
               const uint16_t *__restrict__ q, uint16_t *__restrict__ out,
               const int32_t *__restrict__ qo_indptr, const int32_t *__restrict__ prefix_lens,
               const int32_t *__restrict__ bt, int bt_stride, int hkv, int group, int num_pages,
               float scale_log2, int paired, int n_hgroups) {
    __shared__ __attribute__((aligned(1024))) uint16_t s_k[2 * TILE];
    __shared__ __attribute__((aligned(1024))) uint16_t s_v[2 * TILE];
    __shared__ int32_t s_bt[kBtCache];
    prefill_block<kTableInLds, NW>(kpool, vpool, q, out, qo_indptr, prefix_lens, bt, bt_stride, hkv, group, num_pages,
                               scale_log2, paired, n_hgroups, blockIdx.x, blockIdx.y, s_k, s_v, s_bt);
}

// Key-range split of small grids (4-wave blocks): work-group (x, b) runs
// piece x % max_pieces of block unit x / max_pieces (nothing when the block
// has fewer pieces), so the pieces of a block are dispatched together,
// heaviest blocks first.
template <bool kTableInLds>
__global__ void __launch_bounds__(256, 2)
k_prefill_split(const uint16_t *__restrict__ kpool, const uint16_t *__restrict__ vpool,
                const uint16_t *__restrict__ q, uint16_t *__restrict__ out,
                const int32_t *__restrict__ qo_indptr, const int32_t *__restrict__ prefix_lens,
                const int32_t *__restrict__ bt, int bt_stride, int hkv, int group, int num_pages,
                float scale_log2, int n_hgroups, float *__restrict__ ws_o, float2 *__restrict__ ws_ml,
                int64_t rows, int piece_tiles, int max_pieces) {
    __shared__ __attribute__((aligned(1024))) uint16_t s_k[2 * TILE];
    __shared__ __attribute__((aligned(1024))) uint16_t s_v[2 * TILE];
    __shared__ int32_t s_bt[kBtCache];
    const int unit = static_cast<int>(blockIdx.x) / max_pieces;
    const SplitOut sp{ws_o, ws_ml, rows, piece_tiles, max_pieces, static_cast<int>(blockIdx.x) % max_pieces};
    prefill_block<kTableInLds, 4, true>(kpool, vpool, q, out, qo_indptr, prefix_lens, bt, bt_stride, hkv, group,
                                        num_pages, scale_log2, 0, n_hgroups, unit, blockIdx.y, s_k, s_v, s_bt, sp);
}

// Merge of the pieces of every split block: work-group (q * hq + h, b) takes
// the 32 rows of block q of sequence b for query head h (8 threads per row,
// 16 dims each): with M the largest reference maximum of the pieces,
// O = sum_i 2^(m_i - M) O~_i / sum_i 2^(m_i - M) l_i, written as bf16.
// Blocks with one piece were written by the split kernel itself.
__global__ void __launch_bounds__(256)
k_prefill_merge(const float *__restrict__ ws_o, const float2 *__restrict__ ws_ml, uint16_t *__restrict__ out,
                const int32_t *__restrict__ qo_indptr, const int32_t *__restrict__ prefix_lens, int hq,
                int64_t rows, int piece_tiles, int max_pieces) {
    const int b = blockIdx.y;
    const int qb = blockIdx.x / hq, h = blockIdx.x % hq;
    const int row0 = qo_indptr[b];
    const int n = qo_indptr[b + 1] - row0;
    if (32 * qb >= n) return;
    const int k = prefill_pieces(prefill_block_tiles(prefix_lens[b], n, qb), piece_tiles, max_pieces);
    if (k < 2) return;
    const int i = 32 * qb + static_cast<int>(threadIdx.x >> 3);
    if (i >= n) return;
    const int d0 = 16 * (threadIdx.x & 7);
    const size_t row = static_cast<size_t>(row0 + i) * hq + h;
    const size_t stride = static_cast<size_t>(rows) * hq;  // one piece's slot
    float m = -INFINITY;
    for (int p = 0; p < k; ++p) m = fmaxf(m, ws_ml[p * stride + row].x);
    float l = 0.f, o[16];
#pragma unroll
    for (int e = 0; e < 16; ++e) o[e] = 0.f;
    for (int p = 0; p < k; ++p) {
        const float2 ml = ws_ml[p * stride + row];
        if (!(ml.y > 0.f)) continue;  // no keys: contributes nothing
        const float w = exp2f(ml.x - m);
        l += w * ml.y;
        const float4 *src = reinterpret_cast<const float4 *>(ws_o + (p * stride + row) * kHeadDim + d0);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const float4 v = src[e];
            o[4 * e + 0] += w * v.x;
            o[4 * e + 1] += w * v.y;
            o[4 * e + 2] += w * v.z;
            o[4 * e + 3] += w * v.w;
        }
    }
    const float inv = 1.f / l;
    uint32_t packed[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) packed[e] = cvt2(o[2 * e] * inv, o[2 * e + 1] * inv);
    uint4 *dst = reinterpret_cast<uint4 *>(out + row * kHeadDim + d0);
    dst[0] = make_uint4(packed[0], packed[1], packed[2], packed[3]);
    dst[1] = make_uint4(packed[4], packed[5], packed[6], packed[7]);
}

}  // namespace

namespace mw {

void prefill_split_plan(int32_t batch, const int32_t *h_new_lens, const int32_t *h_prefix_lens, int hq,
                        int64_t cus, PrefillPlan *p) {
    p->pieces = 1;
    p->piece_tiles = 0;
    p->split_bytes = 0;
    p->rows = 0;
    int max_nt = 0;
    int64_t units = 0;  // 32-position query blocks x kv heads x head groups
    for (int32_t b = 0; b < batch; ++b) {
        const int n = h_new_lens[b], r = h_prefix_lens[b];
        p->rows += n;
        if (n > 0) max_nt = std::max(max_nt, prefill_block_tiles(r, n, (n - 1) / 32));
        units += (n + 31) / 32;
    }
    units *= static_cast<int64_t>(p->hkv) * p->n_hgroups;
    if (p->waves != 4 || units == 0) return;
    const auto bytes_for = [&](int pieces) {
        return pieces > 1 ? static_cast<size_t>(pieces) * p->rows * hq * (kHeadDim * 4 + 8) : 0;
    };
    if (cus <= 0) {  // sizing: the most pieces any stream's plan can take
        p->piece_tiles = kPrefillMinPieceTiles;
        p->pieces = prefill_pieces(max_nt, kPrefillMinPieceTiles, kPrefillMaxPieces);
        p->split_bytes = bytes_for(p->pieces);
        return;
    }
    // Measured on 2048-token chunks of a one-kv-head shard and of an 8-kv-head
    // layer (piece lengths swept 4..48 tiles): with fewer blocks than CUs,
    // pieces that give about two work-groups per CU (the longest block cut in
    // 2C / units); with fewer than two per CU, long blocks (96 tiles and more)
    // cut in three, which evens out the CUs holding one block and those
    // holding two; otherwise (short blocks, or a grid of two blocks per CU) the
    // merge pass costs more than the cut saves.
    int k = 1;
    if (units < cus)
        k = static_cast<int>(std::min<int64_t>(kPrefillMaxPieces, std::max<int64_t>(2, (2 * cus + units - 1) / units)));
    else if (units < 2 * cus && max_nt >= 96)
        k = 3;
    const int best_pt = k > 1 ? std::max(kPrefillMinPieceTiles, (max_nt + k - 1) / k) : 0;
    if (best_pt == 0) return;
    p->piece_tiles = best_pt;
    p->pieces = prefill_pieces(max_nt, best_pt, kPrefillMaxPieces);
    p->split_bytes = bytes_for(p->pieces);
}



// Pairs of query blocks of bm positions over a batch's sequences.
static int64_t prefill_pairs(int32_t batch, const int32_t *h_new_lens, int64_t bm) {
    int64_t n_pairs = 0;
    for (int32_t b = 0; b < batch; ++b) n_pairs += ((h_new_lens[b] + bm - 1) / bm + 1) / 2;
    return n_pairs;
}

mw_status prefill_prepare(const mw_prefill_args *a, int64_t cus, bool allow_small, PrefillPlan *p, const char *who) {
    if (!a || !a->pool || a->batch < 0 || a->batch > 65535 || a->bt_stride < 1 ||
        (a->batch > 0 && (!a->h_new_lens || !a->h_prefix_lens)))
        return fail(MW_ERR_INVALID_ARG, "%s: bad arguments", who);
    const mw_attn_shape *shape = &a->shape;
    const mw_kv_pool *pool = a->pool;
    if (shape->head_dim != kHeadDim) return fail(MW_ERR_UNSUPPORTED, "%s: head_dim must be 128", who);
    if (!(shape->scale > 0.f) || !(shape->scale < INFINITY))
        return fail(MW_ERR_INVALID_ARG, "%s: scale must be positive and finite", who);
    if (shape->num_kv_heads != pool->desc.num_kv_heads || shape->num_q_heads < 1 ||
        shape->num_q_heads % shape->num_kv_heads)
        return fail(MW_ERR_INVALID_ARG, "%s: num_q_heads must be a multiple of the pool's %d kv heads", who,
                    pool->desc.num_kv_heads);
    int64_t max_n = 0, max_pages = 0;
    for (int32_t b = 0; b < a->batch; ++b) {
        const int32_t n = a->h_new_lens[b], r = a->h_prefix_lens[b];
        if (n < 0 || r < 0 || static_cast<int64_t>(n) + r > static_cast<int64_t>(a->bt_stride) * kPageSize)
            return fail(MW_ERR_INVALID_ARG, "%s: sequence %d: prefix %d + new %d exceeds %d table pages", who, b, r,
                        n, a->bt_stride);
        max_n = n > max_n ? n : max_n;
        const int64_t pages = (static_cast<int64_t>(n) + r + kPageSize - 1) / kPageSize;
        max_pages = pages > max_pages ? pages : max_pages;
    }
    if (max_n > 0 && (!a->d_qo_indptr || !a->d_prefix_lens || !a->d_block_table || !a->d_q || !a->d_out))
        return fail(MW_ERR_INVALID_ARG, "%s: NULL device pointer", who);
    if (max_n > 0 && (!aligned16(a->d_q) || !aligned16(a->d_out)))
        return fail(MW_ERR_INVALID_ARG, "%s: Q and O must be 16-byte aligned", who);
    prefill_plan_lengths(a->batch, a->h_new_lens, shape->num_kv_heads, shape->num_q_heads / shape->num_kv_heads, cus,
                         allow_small, p);
    p->table_in_lds = max_pages <= kBtCache;
    p->scale_log2 = shape->scale * kLog2e;
    if (p->gx > 0x7fffffff) return fail(MW_ERR_UNSUPPORTED, "%s: grid too large", who);
    return MW_OK;
}

void prefill_plan_lengths(int32_t batch, const int32_t *h_new_lens, int hkv, int group, int64_t cus,
                          bool allow_small, PrefillPlan *p) {
    p->hkv = hkv;
    p->group = group;
    p->n_hgroups = (group + 3) / 4;
    p->batch = batch;
    p->table_in_lds = true;
    p->scale_log2 = 0.f;
    p->paired = 0;
    p->gx = 0;
    p->pieces = 1;
    p->piece_tiles = 0;
    p->rows = 0;
    p->split_bytes = 0;
    p->waves = 8;
    int64_t max_n = 0;
    for (int32_t b = 0; b < batch; ++b) max_n = std::max<int64_t>(max_n, h_new_lens[b]);
    if (max_n == 0) return;
    auto pairs_of = [&](int64_t bm) { return prefill_pairs(batch, h_new_lens, bm) * p->hkv * p->n_hgroups; };
    // Eight waves (64-position blocks, one work-group per CU) unless their pairs
    // would not even give every CU one: then four waves (32-position blocks,
    // two work-groups per CU), which doubles the work-groups.
    int64_t bm = BM, slots = cus;
    if (allow_small && pairs_of(BM) < cus) {
        p->waves = 4;
        bm = BM / 2;
        slots = 2 * cus;
    }
    // Pair blocks only when the pairs fill whole rounds of the work-group slots
    // of the stream's CUs: equal-cost pairs then finish together.  Otherwise
    // single blocks, heaviest first, fill the last round better.
    const int64_t max_qblocks = (max_n + bm - 1) / bm;
    const int64_t n_pairs = pairs_of(bm);
    const int64_t rounds = (n_pairs + slots - 1) / slots;
    p->paired = n_pairs >= slots && rounds * slots * 20 <= n_pairs * 21;
    p->gx = (p->paired ? (max_qblocks + 1) / 2 : max_qblocks) * p->hkv * p->n_hgroups;
}

}  // namespace mw

extern "C" mw_status mw_prefill_attn(const mw_kv_pool *pool, const mw_attn_shape *shape, int32_t batch,
                                     const int32_t *h_new_lens, const int32_t *h_prefix_lens,
                                     const int32_t *d_qo_indptr, const int32_t *d_prefix_lens,
                                     const int32_t *d_block_table, int32_t bt_stride, const void *d_q,
                                     void *d_out, mw_stream stream, mw_timing *timing) {
    const char *who = "mw_prefill_attn";
    if (!shape) return fail(MW_ERR_INVALID_ARG, "%s: bad arguments", who);
    const mw_prefill_args a{pool,          *shape,        batch,     h_new_lens, h_prefix_lens, d_qo_indptr,
                            d_prefix_lens, d_block_table, bt_stride, d_q,        d_out};
    hipStream_t s = static_cast<hipStream_t>(stream);
    PrefillPlan pl;
    mw_status st = prefill_prepare(&a, stream_cus(s), true, &pl, who);
    if (st != MW_OK) return st;
    st = timing_begin(timing, s);
    if (st != MW_OK) return st;
    if (pl.gx > 0) {
        auto kernel = pl.waves == 4 ? (pl.table_in_lds ? k_prefill_attn<true, 4> : k_prefill_attn<false, 4>)
                                    : (pl.table_in_lds ? k_prefill_attn<true, 8> : k_prefill_attn<false, 8>);
        hipLaunchKernelGGL(kernel, dim3(static_cast<unsigned>(pl.gx), batch), dim3(64 * pl.waves), 0, s, pool->k,
                           pool->v, static_cast<const uint16_t *>(d_q), static_cast<uint16_t *>(d_out), d_qo_indptr,
                           d_prefix_lens, d_block_table, bt_stride, pl.hkv, pl.group, pool->desc.num_pages,
                           pl.scale_log2, pl.paired, pl.n_hgroups);
        st = check_launch("k_prefill_attn");
        if (st != MW_OK) return st;
    }
    st = timing_kernel_done(timing, s);
    timing_end(timing);
    return st;
}

extern "C" mw_status mw_prefill_workspace_size(const mw_attn_shape *shape, int32_t batch, const int32_t *h_new_lens,
                                               const int32_t *h_prefix_lens, int32_t num_cus, size_t *bytes) {
    const char *who = "mw_prefill_workspace_size";
    if (!shape || !bytes || batch < 0 || batch > 65535 || num_cus < 0 || (batch > 0 && (!h_new_lens || !h_prefix_lens)))
        return fail(MW_ERR_INVALID_ARG, "%s: bad arguments", who);
    if (shape->head_dim != kHeadDim) return fail(MW_ERR_UNSUPPORTED, "%s: head_dim must be 128", who);
    if (shape->num_kv_heads < 1 || shape->num_q_heads < 1 || shape->num_q_heads % shape->num_kv_heads)
        return fail(MW_ERR_INVALID_ARG, "%s: num_q_heads must be a multiple of num_kv_heads", who);
    for (int32_t b = 0; b < batch; ++b)
        if (h_new_lens[b] < 0 || h_prefix_lens[b] < 0 ||
            static_cast<int64_t>(h_new_lens[b]) + h_prefix_lens[b] > INT32_MAX - 64)
            return fail(MW_ERR_INVALID_ARG, "%s: sequence %d: bad lengths", who, b);
    PrefillPlan pl{};
    pl.hkv = shape->num_kv_heads;
    pl.group = shape->num_q_heads / pl.hkv;
    pl.n_hgroups = (pl.group + 3) / 4;
    // the split runs where the launch takes 4-wave blocks (as in prefill_prepare);
    // without a CU count, size for any stream
    pl.waves = num_cus == 0 || prefill_pairs(batch, h_new_lens, BM) * pl.hkv * pl.n_hgroups < num_cus ? 4 : 8;
    prefill_split_plan(batch, h_new_lens, h_prefix_lens, shape->num_q_heads, num_cus, &pl);
    *bytes = pl.split_bytes;
    return MW_OK;
}

extern "C" mw_status mw_prefill_attn_ws(const mw_kv_pool *pool, const mw_attn_shape *shape, int32_t batch,
                                        const int32_t *h_new_lens, const int32_t *h_prefix_lens,
                                        const int32_t *d_qo_indptr, const int32_t *d_prefix_lens,
                                        const int32_t *d_block_table, int32_t bt_stride, const void *d_q,
                                        void *d_out, void *d_workspace, size_t workspace_bytes, mw_stream stream,
                                        mw_timing *timing) {
    const char *who = "mw_prefill_attn_ws";
    if (!shape) return fail(MW_ERR_INVALID_ARG, "%s: bad arguments", who);
    const mw_prefill_args a{pool,          *shape,        batch,     h_new_lens, h_prefix_lens, d_qo_indptr,
                            d_prefix_lens, d_block_table, bt_stride, d_q,        d_out};
    hipStream_t s = static_cast<hipStream_t>(stream);
    PrefillPlan pl;
    const int64_t cus = stream_cus(s);
    mw_status st = prefill_prepare(&a, cus, true, &pl, who);
    if (st != MW_OK) return st;
    prefill_split_plan(batch, h_new_lens, h_prefix_lens, shape->num_q_heads, cus, &pl);
    if (pl.pieces < 2 || pl.gx == 0) return mw_prefill_attn(pool, shape, batch, h_new_lens, h_prefix_lens,
                                                            d_qo_indptr, d_prefix_lens, d_block_table, bt_stride,
                                                            d_q, d_out, stream, timing);
    if (!d_workspace || !aligned16(d_workspace) || workspace_bytes < pl.split_bytes)
        return fail(MW_ERR_INVALID_ARG, "%s: the split needs a 16-byte aligned workspace of %zu bytes (got %zu)",
                    who, pl.split_bytes, workspace_bytes);
    int max_n = 0;
    for (int32_t b = 0; b < batch; ++b) max_n = h_new_lens[b] > max_n ? h_new_lens[b] : max_n;
    const int64_t gx = static_cast<int64_t>((max_n + 31) / 32) * pl.hkv * pl.n_hgroups;  // single blocks
    if (gx * pl.pieces > 0x7fffffff) return fail(MW_ERR_UNSUPPORTED, "%s: grid too large", who);
    st = timing_begin(timing, s);
    if (st != MW_OK) return st;
    float *ws_o = static_cast<float *>(d_workspace);
    float2 *ws_ml = reinterpret_cast<float2 *>(static_cast<char *>(d_workspace) +
                                               static_cast<size_t>(pl.pieces) * pl.rows * shape->num_q_heads *
                                                   kHeadDim * 4);
    auto kernel = pl.table_in_lds ? k_prefill_split<true> : k_prefill_split<false>;
    hipLaunchKernelGGL(kernel, dim3(static_cast<unsigned>(gx * pl.pieces), batch), dim3(256), 0, s, pool->k,
                       pool->v, static_cast<const uint16_t *>(d_q), static_cast<uint16_t *>(d_out), d_qo_indptr,
                       d_prefix_lens, d_block_table, bt_stride, pl.hkv, pl.group, pool->desc.num_pages, pl.scale_log2,
                       pl.n_hgroups, ws_o, ws_ml, pl.rows, pl.piece_tiles, pl.pieces);
    st = check_launch("k_prefill_split");
    if (st != MW_OK) return st;
    st = timing_kernel_done(timing, s);
    if (st != MW_OK) return st;
    const int64_t gm = static_cast<int64_t>((max_n + 31) / 32) * shape->num_q_heads;
    hipLaunchKernelGGL(k_prefill_merge, dim3(static_cast<unsigned>(gm), batch), dim3(256), 0, s, ws_o, ws_ml,
                       static_cast<uint16_t *>(d_out), d_qo_indptr, d_prefix_lens, shape->num_q_heads, pl.rows,
                       pl.piece_tiles, pl.pieces);
    st = check_launch("k_prefill_merge");
    if (st != MW_OK) return st;
    st = timing_kernel_done(timing, s);
    timing_end(timing);
    return st;
}
