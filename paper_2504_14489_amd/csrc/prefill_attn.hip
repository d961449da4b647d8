// Causal prefill attention of a chunk of new tokens over its cached prefix:
// the kernel (its work-group body is in prefill_block.h) and its launch.
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

}  // namespace

namespace mw {

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
    p->hkv = shape->num_kv_heads;
    p->group = shape->num_q_heads / p->hkv;
    p->n_hgroups = (p->group + 3) / 4;
    p->batch = a->batch;
    p->table_in_lds = max_pages <= kBtCache;
    p->scale_log2 = shape->scale * kLog2e;
    p->paired = 0;
    p->gx = 0;
    p->waves = 8;
    if (max_n == 0) return MW_OK;
    auto pairs_of = [&](int64_t bm) {
        int64_t n_pairs = 0;
        for (int32_t b = 0; b < a->batch; ++b) n_pairs += ((a->h_new_lens[b] + bm - 1) / bm + 1) / 2;
        return n_pairs * p->hkv * p->n_hgroups;
    };
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
    if (p->gx > 0x7fffffff) return fail(MW_ERR_UNSUPPORTED, "%s: grid too large", who);
    return MW_OK;
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
