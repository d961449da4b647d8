// Paged KV pool: host-side page allocator and the append / gather kernels.
//
// The pool is one [num_pages][num_kv_heads][page_size][head_dim] bf16 array
// for K and one for V.  A (page, kv-head) block is 16 x 128 bf16 = 4 KiB
// contiguous, so a token's row for one head is 256 contiguous bytes and every
// copy below moves whole 16-byte vectors.
#include "mw_internal.h"

using namespace mw;

namespace {

constexpr int kVecPerRow = kHeadDim * 2 / 16;  // 16-byte vectors per (token, head) row

// Copies new K/V rows [rows][hkv][128] into their page slots.
// grid.y = sequence; grid.x strides over that sequence's (token, head, vector).
__global__ void __launch_bounds__(256)
k_kv_write(uint4 *__restrict__ kpool, uint4 *__restrict__ vpool, const uint4 *__restrict__ knew,
           const uint4 *__restrict__ vnew, const int32_t *__restrict__ qo_indptr,
           const int32_t *__restrict__ start_pos, const int32_t *__restrict__ bt, int bt_stride,
           int num_pages, int hkv) {
    const int b = blockIdx.y;
    const int row0 = qo_indptr[b];
    const int n = qo_indptr[b + 1] - row0;
    const int pos0 = start_pos[b];
    const int per_tok = hkv * kVecPerRow;
    const int total = n * per_tok;
    const int32_t *btrow = bt + static_cast<size_t>(b) * bt_stride;
    for (int idx = blockIdx.x * blockDim.x + threadIdx.x; idx < total;
         idx += gridDim.x * blockDim.x) {
        const int i = idx / per_tok;
        const int rem = idx - i * per_tok;
        const int h = rem / kVecPerRow;
        const int c = rem - h * kVecPerRow;
        const int pos = pos0 + i;
        if (pos < 0 || pos >= bt_stride * kPageSize) continue;
        const int page = btrow[pos / kPageSize];
        if (page < 0 || page >= num_pages) continue;
        const size_t dst =
            ((static_cast<size_t>(page) * hkv + h) * kPageSize + (pos % kPageSize)) * kVecPerRow + c;
        const size_t src = (static_cast<size_t>(row0 + i) * hkv + h) * kVecPerRow + c;
        kpool[dst] = knew[src];
        vpool[dst] = vnew[src];
    }
}

// Gathers tokens [0, n_tokens) of one sequence into [n_tokens][hkv][128].
__global__ void __launch_bounds__(256)
k_kv_gather(const uint4 *__restrict__ kpool, const uint4 *__restrict__ vpool,
            uint4 *__restrict__ kout, uint4 *__restrict__ vout, const int32_t *__restrict__ bt,
            int n_tokens, int num_pages, int hkv) {
    const int per_tok = hkv * kVecPerRow;
    const int total = n_tokens * per_tok;
    for (int idx = blockIdx.x * blockDim.x + threadIdx.x; idx < total;
         idx += gridDim.x * blockDim.x) {
        const int t = idx / per_tok;
        const int rem = idx - t * per_tok;
        const int h = rem / kVecPerRow;
        const int c = rem - h * kVecPerRow;
        const int page = bt[t / kPageSize];
        uint4 kv = make_uint4(0, 0, 0, 0), vv = make_uint4(0, 0, 0, 0);
        if (page >= 0 && page < num_pages) {
            const size_t src =
                ((static_cast<size_t>(page) * hkv + h) * kPageSize + (t % kPageSize)) * kVecPerRow + c;
            kv = kpool[src];
            vv = vpool[src];
        }
        kout[idx] = kv;
        vout[idx] = vv;
    }
}

}  // namespace

extern "C" {

mw_status mw_kv_pool_create(const mw_kv_pool_desc *desc, void *d_k_pages, void *d_v_pages,
                            mw_kv_pool **out) {
    if (!desc || !out || !d_k_pages || !d_v_pages)
        return fail(MW_ERR_INVALID_ARG, "mw_kv_pool_create: NULL argument");
    if (desc->num_pages < 1 || desc->num_kv_heads < 1)
        return fail(MW_ERR_INVALID_ARG, "mw_kv_pool_create: num_pages and num_kv_heads must be >= 1");
    if (desc->page_size != kPageSize || desc->head_dim != kHeadDim)
        return fail(MW_ERR_UNSUPPORTED, "mw_kv_pool_create: only page_size 16 and head_dim 128");
    if (!aligned16(d_k_pages) || !aligned16(d_v_pages))
        return fail(MW_ERR_INVALID_ARG, "mw_kv_pool_create: pool arrays must be 16-byte aligned");
    mw_kv_pool *p = new (std::nothrow) mw_kv_pool();
    if (!p) return fail(MW_ERR_INVALID_ARG, "mw_kv_pool_create: out of host memory");
    p->desc = *desc;
    p->k = static_cast<uint16_t *>(d_k_pages);
    p->v = static_cast<uint16_t *>(d_v_pages);
    p->is_free.assign(desc->num_pages, 1);
    for (int32_t i = 0; i < desc->num_pages; ++i) p->free_list.push_back(i);
    *out = p;
    return MW_OK;
}

mw_status mw_kv_pool_destroy(mw_kv_pool *pool) {
    delete pool;
    return MW_OK;
}

mw_status mw_kv_pool_set_free_order(mw_kv_pool *pool, const int32_t *perm, int32_t n) {
    if (!pool || (n > 0 && !perm) || n < 0)
        return fail(MW_ERR_INVALID_ARG, "mw_kv_pool_set_free_order: bad arguments");
    std::vector<uint8_t> seen(pool->desc.num_pages, 0);
    for (int32_t i = 0; i < n; ++i) {
        if (perm[i] < 0 || perm[i] >= pool->desc.num_pages || seen[perm[i]])
            return fail(MW_ERR_INVALID_ARG,
                        "mw_kv_pool_set_free_order: entry %d (%d) is out of range or repeated", i,
                        perm[i]);
        seen[perm[i]] = 1;
    }
    pool->free_list.assign(perm, perm + n);
    pool->is_free = seen;
    return MW_OK;
}

mw_status mw_kv_pool_alloc(mw_kv_pool *pool, int32_t n_pages, int32_t *pages_out) {
    if (!pool || n_pages < 0 || (n_pages > 0 && !pages_out))
        return fail(MW_ERR_INVALID_ARG, "mw_kv_pool_alloc: bad arguments");
    if (static_cast<size_t>(n_pages) > pool->free_list.size())
        return fail(MW_ERR_OUT_OF_PAGES, "mw_kv_pool_alloc: %d pages requested, %zu free", n_pages,
                    pool->free_list.size());
    for (int32_t i = 0; i < n_pages; ++i) {
        pages_out[i] = pool->free_list.front();
        pool->free_list.pop_front();
        pool->is_free[pages_out[i]] = 0;
    }
    return MW_OK;
}

mw_status mw_kv_pool_free(mw_kv_pool *pool, const int32_t *pages, int32_t n_pages) {
    if (!pool || n_pages < 0 || (n_pages > 0 && !pages))
        return fail(MW_ERR_INVALID_ARG, "mw_kv_pool_free: bad arguments");
    std::vector<uint8_t> mark(pool->is_free);
    for (int32_t i = 0; i < n_pages; ++i) {
        if (pages[i] < 0 || pages[i] >= pool->desc.num_pages || mark[pages[i]])
            return fail(MW_ERR_INVALID_ARG, "mw_kv_pool_free: page %d is out of range or already free",
                        pages[i]);
        mark[pages[i]] = 1;
    }
    for (int32_t i = 0; i < n_pages; ++i) pool->free_list.push_back(pages[i]);
    pool->is_free.swap(mark);
    return MW_OK;
}

mw_status mw_kv_pool_num_free(const mw_kv_pool *pool, int32_t *n_free) {
    if (!pool || !n_free) return fail(MW_ERR_INVALID_ARG, "mw_kv_pool_num_free: NULL argument");
    *n_free = static_cast<int32_t>(pool->free_list.size());
    return MW_OK;
}

mw_status mw_kv_pool_write(const mw_kv_pool *pool, int32_t batch, const int32_t *h_new_lens,
                           const int32_t *h_start_pos, const int32_t *d_qo_indptr,
                           const int32_t *d_start_pos, const int32_t *d_block_table,
                           int32_t bt_stride, const void *d_k_new, const void *d_v_new,
                           mw_stream stream, mw_timing *timing) {
    if (!pool || batch < 0 || (batch > 0 && (!h_new_lens || !h_start_pos || !d_qo_indptr ||
                                             !d_start_pos || !d_block_table)) ||
        bt_stride < 1 || batch > 65535)
        return fail(MW_ERR_INVALID_ARG, "mw_kv_pool_write: bad arguments");
    int64_t max_n = 0, total = 0;
    for (int32_t b = 0; b < batch; ++b) {
        if (h_new_lens[b] < 0 || h_start_pos[b] < 0 ||
            static_cast<int64_t>(h_start_pos[b]) + h_new_lens[b] >
                static_cast<int64_t>(bt_stride) * kPageSize)
            return fail(MW_ERR_INVALID_ARG,
                        "mw_kv_pool_write: sequence %d writes positions [%d, %d) beyond its table "
                        "of %d pages",
                        b, h_start_pos[b], h_start_pos[b] + h_new_lens[b], bt_stride);
        max_n = h_new_lens[b] > max_n ? h_new_lens[b] : max_n;
        total += h_new_lens[b];
    }
    if (total > 0 && (!d_k_new || !d_v_new || !aligned16(d_k_new) || !aligned16(d_v_new)))
        return fail(MW_ERR_INVALID_ARG, "mw_kv_pool_write: new K/V must be 16-byte aligned");
    hipStream_t s = static_cast<hipStream_t>(stream);
    mw_status st = timing_begin(timing, s);
    if (st != MW_OK) return st;
    if (total > 0) {
        const int per_tok = pool->desc.num_kv_heads * kVecPerRow;
        int64_t blocks = (max_n * per_tok + 255) / 256;
        if (blocks > 4096) blocks = 4096;
        hipLaunchKernelGGL(k_kv_write, dim3(static_cast<unsigned>(blocks), batch), dim3(256), 0, s,
                           reinterpret_cast<uint4 *>(pool->k), reinterpret_cast<uint4 *>(pool->v),
                           static_cast<const uint4 *>(d_k_new), static_cast<const uint4 *>(d_v_new),
                           d_qo_indptr, d_start_pos, d_block_table, bt_stride, pool->desc.num_pages,
                           pool->desc.num_kv_heads);
        st = check_launch("k_kv_write");
        if (st != MW_OK) return st;
    }
    st = timing_kernel_done(timing, s);
    timing_end(timing);
    return st;
}

mw_status mw_kv_pool_gather(const mw_kv_pool *pool, const int32_t *d_block_table, int32_t n_tokens,
                            void *d_k_out, void *d_v_out, mw_stream stream) {
    if (!pool || n_tokens < 0 || (n_tokens > 0 && (!d_block_table || !d_k_out || !d_v_out)))
        return fail(MW_ERR_INVALID_ARG, "mw_kv_pool_gather: bad arguments");
    if (n_tokens == 0) return MW_OK;
    if (!aligned16(d_k_out) || !aligned16(d_v_out))
        return fail(MW_ERR_INVALID_ARG, "mw_kv_pool_gather: outputs must be 16-byte aligned");
    const int64_t per_tok = pool->desc.num_kv_heads * kVecPerRow;
    int64_t blocks = (n_tokens * per_tok + 255) / 256;
    if (blocks > 4096) blocks = 4096;
    hipLaunchKernelGGL(k_kv_gather, dim3(static_cast<unsigned>(blocks)), dim3(256), 0,
                       static_cast<hipStream_t>(stream), reinterpret_cast<const uint4 *>(pool->k),
                       reinterpret_cast<const uint4 *>(pool->v), static_cast<uint4 *>(d_k_out),
                       static_cast<uint4 *>(d_v_out), d_block_table, n_tokens, pool->desc.num_pages,
                       pool->desc.num_kv_heads);
    return check_launch("k_kv_gather");
}

}  // extern "C"
