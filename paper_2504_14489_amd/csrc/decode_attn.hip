// Decode attention: one query token per sequence over its paged context --
// the balanced split kernel, which merges its own split segments, the
// fixed-chunk split kernel and its combine kernel (their bodies are in
// decode_block.h), and their launch.
#include <algorithm>
#include <climits>
#include <atomic>
#include <mutex>

#include "decode_block.h"

using namespace mw;

namespace {

using namespace dk;

__global__ void __launch_bounds__(kThreads)
k_decode_split(const uint16_t *__restrict__ kpool, const uint16_t *__restrict__ vpool,
               const uint16_t *__restrict__ q, uint16_t *__restrict__ out,
               const int32_t *__restrict__ seq_lens, const int32_t *__restrict__ bt, int bt_stride,
               float *__restrict__ ws_o, float2 *__restrict__ ws_ml, int32_t *__restrict__ ws_cbase,
               int batch, int hkv, int group, int num_pages, float scale_log2, int ch_pages) {
    __shared__ __attribute__((aligned(16))) uint16_t s_v[kWaves * kWaveBufElems];
    __shared__ float s_m[kWaves][16];
    __shared__ float s_l[kWaves][16];
    decode_unit<false>(kpool, vpool, q, out, seq_lens, bt, bt_stride, ws_o, ws_ml, ws_cbase, batch, hkv, group,
                       num_pages, scale_log2, ch_pages, blockIdx.x, threadIdx.x, s_v, s_m, s_l);
}

// Balanced split: unit u streams pages [u per_unit, (u + 1) per_unit) of the
// batch's (sequence, kv head) segments laid end to end.
__global__ void __launch_bounds__(kThreads)
k_decode_balanced(const uint16_t *__restrict__ kpool, const uint16_t *__restrict__ vpool,
                  const uint16_t *__restrict__ q, uint16_t *__restrict__ out,
                  const int32_t *__restrict__ seq_lens, const int32_t *__restrict__ bt, int bt_stride,
                  float *__restrict__ ws_o, float2 *__restrict__ ws_ml, uint32_t *__restrict__ flags,
                  uint32_t tag, int64_t slots, int batch, int hkv, int group, int num_pages, float scale_log2,
                  int64_t per_unit, int64_t total, int aligned) {
    __shared__ __attribute__((aligned(16))) uint16_t s_v[kWaves * kWaveBufElems];
    __shared__ float s_m[kWaves][16];
    __shared__ float s_l[kWaves][16];
    decode_span(kpool, vpool, q, out, seq_lens, bt, bt_stride, ws_o, ws_ml, flags, tag, slots, batch, hkv, group,
                num_pages, scale_log2, per_unit, total, aligned != 0, blockIdx.x, threadIdx.x, s_v, s_m, s_l);
}

// Combine of the fixed-chunk split: one work-group per (sequence, kv head);
// chunk c of sequence b is in slot (ws_cbase[b] + c) hkv + kv head.  (The
// balanced split merges its segments itself.)
__global__ void __launch_bounds__(kThreads)
k_decode_combine(uint16_t *__restrict__ out, const int32_t *__restrict__ seq_lens,
                 const float *__restrict__ ws_o, const float2 *__restrict__ ws_ml,
                 const int32_t *__restrict__ ws_cbase, int hkv, int group, int ch_pages, int bt_stride,
                 int64_t slots) {
    const int b = blockIdx.x / hkv, kvh = blockIdx.x % hkv;
    const int nch = chunks_of(seq_lens[b], ch_pages, bt_stride);
    const int64_t first = static_cast<int64_t>(ws_cbase[b]) * hkv + kvh;
    if (nch <= 1) return;  // written by the split kernel
    // lengths on the device that disagree with the host copy must not lead
    // outside the workspace
    if (first < 0 || first + static_cast<int64_t>(nch - 1) * hkv >= slots) return;
    merge_pieces(out, ws_o, ws_ml, first, hkv, nch, b, hkv, kvh, group, threadIdx.x);
}

// Balanced split: units per CU of the stream (two 4-wave work-groups fit a
// CU), the most units (two per CU of a 256-CU device; the workspace is sized
// for it) and the fewest pages a unit streams (two pairs per wave: short
// calls are bound by latency, not bytes, and fewer, longer pieces leave less
// to merge at the end).
constexpr int64_t kBalancedPerCu = 2;
constexpr int64_t kBalancedMaxUnits = 512;
constexpr int64_t kBalancedMinPages = 16;

struct Plan {
    int64_t units;            // work-groups of the split kernel
    int chunk_pages;          // fixed chunks; 0 with the balanced split
    int64_t per_unit, total;  // balanced split: pages per unit, pages in all (of the split's numbering)
    bool aligned;             // balanced split: segments padded to multiples of per_unit
    int64_t slots;            // partial slots of the workspace
    size_t off_ml, off_meta, bytes;
};

size_t align256(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }

// Workspace: partial O [slots][group][128] and (m, l) [slots][group] in fp32,
// then the fixed-chunk split's per-sequence chunk bases or the balanced
// split's per-slot done flags.
void plan_layout(Plan *plan, int32_t batch, int group) {
    const size_t o_bytes = align256(static_cast<size_t>(plan->slots) * group * kHeadDim * 4);
    const size_t ml_bytes = align256(static_cast<size_t>(plan->slots) * group * 8);
    plan->off_ml = o_bytes;
    plan->off_meta = o_bytes + ml_bytes;
    const size_t meta = plan->per_unit > 0 ? static_cast<size_t>(plan->slots) * 4 : static_cast<size_t>(batch) * 4 + 4;
    plan->bytes = plan->off_meta + align256(meta);
}

// chunk_pages > 0: fixed chunks of that many pages; -1 (or 0 with cus = 0):
// automatic fixed chunks; 0 with cus > 0: the balanced split over cus CUs
// (cus < 0: the largest balanced split, for sizing a workspace).
mw_status plan_decode(const mw_attn_shape *shape, int32_t batch, const int32_t *h_seq_lens,
                      int32_t chunk_pages, int32_t bt_stride, int64_t cus, Plan *plan, const char *who) {
    if (!shape || batch < 0 || (batch > 0 && !h_seq_lens))
        return fail(MW_ERR_INVALID_ARG, "%s: bad arguments", who);
    if (shape->head_dim != kHeadDim) return fail(MW_ERR_UNSUPPORTED, "%s: head_dim must be 128", who);
    if (shape->num_kv_heads < 1 || shape->num_q_heads < 1 || shape->num_q_heads % shape->num_kv_heads)
        return fail(MW_ERR_INVALID_ARG, "%s: num_q_heads must be a positive multiple of num_kv_heads", who);
    if (shape->num_q_heads / shape->num_kv_heads > 16)
        return fail(MW_ERR_UNSUPPORTED, "%s: at most 16 query heads per kv head", who);
    if (chunk_pages != 0 && chunk_pages != -1 && (chunk_pages < 8 || chunk_pages > 256 || chunk_pages % 8))
        return fail(MW_ERR_UNSUPPORTED, "%s: chunk_pages must be a multiple of 8 in [8, 256] (or 0, -1)", who);
    for (int32_t b = 0; b < batch; ++b) {
        const int32_t L = h_seq_lens[b];
        if (L < 1 || (bt_stride > 0 && static_cast<int64_t>(L) > static_cast<int64_t>(bt_stride) * kPageSize))
            return fail(MW_ERR_INVALID_ARG, "%s: sequence %d has length %d (table holds %d pages)", who, b,
                        L, bt_stride);
    }
    auto count = [&](int ch) {
        int64_t n = 0;
        for (int32_t b = 0; b < batch; ++b) n += ((h_seq_lens[b] + kPageSize - 1) / kPageSize + ch - 1) / ch;
        return n;
    };
    const int group = shape->num_q_heads / shape->num_kv_heads;
    const int64_t hkv = shape->num_kv_heads;
    auto fixed = [&](int ch, Plan *pl) {
        if (ch <= 0) {
            ch = kAutoChunks[2];
            for (int c : kAutoChunks)
                if (count(c) * hkv >= kAutoMinUnits) {
                    ch = c;
                    break;
                }
        }
        pl->chunk_pages = ch;
        pl->units = pl->slots = count(ch) * hkv;
        pl->per_unit = pl->total = 0;
        pl->aligned = false;
        plan_layout(pl, batch, group);
    };
    // may_align = false for workspace sizing: an aligned split needs no more
    // units than the unaligned one on as many CUs, whose count only grows with
    // the CUs
    auto balanced = [&](int64_t n_cus, Plan *pl, bool may_align) {
        pl->chunk_pages = 0;
        pl->total = count(1) * hkv;
        int64_t units = std::min(kBalancedPerCu * std::max<int64_t>(n_cus, 1), kBalancedMaxUnits);
        units = std::max<int64_t>(1, std::min(units, (pl->total + kBalancedMinPages - 1) / kBalancedMinPages));
        pl->per_unit = std::max<int64_t>(1, (pl->total + units - 1) / units);
        // Few long segments (each cut into two pieces or more): pad every
        // segment to a multiple of the range, so that a unit holds one piece
        // of one segment (a range that straddles two segments costs a second
        // piece set-up and a second merge at the end).  The range is the
        // shortest one, no shorter than the balanced one, whose padded
        // segments need no more units than the balanced split (equal segments
        // are then cut in equal pieces); padding is used only if it keeps at
        // least 90% of those units busy.
        pl->aligned = false;
        int64_t np_min = INT64_MAX, np_max = 0;
        for (int32_t b = 0; b < batch; ++b) {
            const int64_t np = (h_seq_lens[b] + kPageSize - 1) / kPageSize;
            np_min = std::min(np_min, np);
            np_max = std::max(np_max, np);
        }
        const int64_t units_bal = (pl->total + pl->per_unit - 1) / pl->per_unit;
        auto padded_units = [&](int64_t r) {
            int64_t n = 0;
            for (int32_t b = 0; b < batch; ++b) n += ((h_seq_lens[b] + kPageSize - 1) / kPageSize + r - 1) / r;
            return n * hkv;
        };
        if (may_align && batch > 0 && np_min >= 2 * pl->per_unit) {
            int64_t lo = pl->per_unit, hi = np_max;  // padded_units(np_max) = batch * hkv <= units_bal / 2
            while (lo < hi) {
                const int64_t mid = lo + (hi - lo) / 2;
                if (padded_units(mid) <= units_bal)
                    hi = mid;
                else
                    lo = mid + 1;
            }
            const int64_t n = padded_units(lo);
            if (10 * n >= 9 * units_bal) {
                pl->aligned = true;
                pl->per_unit = lo;
                pl->total = n * lo;
            }
        }
        pl->units = pl->total > 0 ? (pl->total + pl->per_unit - 1) / pl->per_unit : 0;
        // piece of unit u of segment s in slot u + s
        pl->slots = pl->units > 0 ? pl->units + static_cast<int64_t>(batch) * hkv - 1 : 0;
        plan_layout(pl, batch, group);
    };
    if (chunk_pages == 0 && cus < 0) {
        // workspace for either split of chunk_pages = 0
        Plan a, b;
        fixed(0, &a);
        balanced(kBalancedMaxUnits, &b, false);
        *plan = a.bytes >= b.bytes ? a : b;
    } else if (chunk_pages == 0 && cus > 0) {
        balanced(cus, plan, true);
    } else {
        fixed(chunk_pages, plan);
    }
    return MW_OK;
}

}  // namespace

namespace mw {

mw_status decode_prepare(const mw_decode_args *a, int64_t cus, DecodePlan *p, const char *who) {
    if (!a || !a->pool || a->bt_stride < 1) return fail(MW_ERR_INVALID_ARG, "%s: bad pool or bt_stride", who);
    const mw_attn_shape *shape = &a->shape;
    Plan pl;
    mw_status st = plan_decode(shape, a->batch, a->h_seq_lens, a->chunk_pages, a->bt_stride, cus, &pl, who);
    if (st != MW_OK) return st;
    if (!(shape->scale > 0.f) || !(shape->scale < INFINITY))
        return fail(MW_ERR_INVALID_ARG, "%s: scale must be positive and finite", who);
    if (shape->num_kv_heads != a->pool->desc.num_kv_heads)
        return fail(MW_ERR_INVALID_ARG, "%s: num_kv_heads %d differs from the pool's %d", who,
                    shape->num_kv_heads, a->pool->desc.num_kv_heads);
    if (a->batch > 0 && (!a->d_seq_lens || !a->d_block_table || !a->d_q || !a->d_out || !a->d_workspace))
        return fail(MW_ERR_INVALID_ARG, "%s: NULL device pointer", who);
    if (a->batch > 0 && (!aligned16(a->d_q) || !aligned16(a->d_out) || !aligned16(a->d_workspace)))
        return fail(MW_ERR_INVALID_ARG, "%s: Q, O and workspace must be 16-byte aligned", who);
    if (a->workspace_bytes < pl.bytes)
        return fail(MW_ERR_INVALID_ARG, "%s: workspace of %zu bytes, %zu needed", who, a->workspace_bytes, pl.bytes);
    if (pl.units > 0x7fffffff) return fail(MW_ERR_UNSUPPORTED, "%s: too many work units", who);
    if (pl.per_unit > 0 && pl.total + pl.units > 0x7fffffff)
        return fail(MW_ERR_UNSUPPORTED, "%s: too many pages for the balanced split", who);
    p->units = pl.units;
    p->chunk_pages = pl.chunk_pages;
    p->per_unit = pl.per_unit;
    p->total = pl.total;
    p->aligned = pl.aligned;
    p->slots = pl.slots;
    p->off_ml = pl.off_ml;
    p->off_meta = pl.off_meta;
    p->bytes = pl.bytes;
    p->hkv = shape->num_kv_heads;
    p->group = shape->num_q_heads / shape->num_kv_heads;
    p->scale_log2 = shape->scale * kLog2e;
    return MW_OK;
}

mw_status decode_combine_launch(const mw_decode_args *a, const DecodePlan &p, hipStream_t s) {
    if (a->batch <= 0) return MW_OK;
    const char *ws = static_cast<const char *>(a->d_workspace);
    hipLaunchKernelGGL(k_decode_combine, dim3(static_cast<unsigned>(a->batch) * p.hkv), dim3(kThreads), 0, s,
                       static_cast<uint16_t *>(a->d_out), a->d_seq_lens, reinterpret_cast<const float *>(ws),
                       reinterpret_cast<const float2 *>(ws + p.off_ml),
                       reinterpret_cast<const int32_t *>(ws + p.off_meta), p.hkv, p.group, p.chunk_pages,
                       a->bt_stride, p.slots);
    return check_launch("k_decode_combine");
}

}  // namespace mw

extern "C" {

mw_status mw_decode_workspace_size(const mw_attn_shape *shape, int32_t batch, const int32_t *h_seq_lens,
                                   int32_t chunk_pages, size_t *bytes) {
    if (!bytes) return fail(MW_ERR_INVALID_ARG, "mw_decode_workspace_size: bytes is NULL");
    Plan pl;
    mw_status st = plan_decode(shape, batch, h_seq_lens, chunk_pages, 0, -1, &pl, "mw_decode_workspace_size");
    if (st != MW_OK) return st;
    *bytes = pl.bytes;
    return MW_OK;
}

}  // extern "C"

namespace {

// Tag of a balanced-split launch, never 0 (the cleared flag value): a done
// flag in a workspace counts only for the launch whose tag it shows.
std::atomic<uint32_t> g_decode_tag{0};
uint32_t next_tag() {
    uint32_t t = 0;
    while (t == 0) t = g_decode_tag.fetch_add(1, std::memory_order_relaxed) + 1;
    return t;
}

// The launches of one planned decode call: the balanced split (which merges
// its own segments), or the fixed-chunk split and its combine.
mw_status decode_launch(const mw_decode_args &a, const DecodePlan &pl, hipStream_t s, mw_timing *timing) {
    const mw_kv_pool *pool = a.pool;
    const int32_t batch = a.batch, bt_stride = a.bt_stride;
    const int32_t *d_seq_lens = a.d_seq_lens, *d_block_table = a.d_block_table;
    const void *d_q = a.d_q;
    void *d_out = a.d_out;
    mw_status st = timing_begin(timing, s);
    if (st != MW_OK) return st;
    if (pl.units > 0) {
        char *ws = static_cast<char *>(a.d_workspace);
        if (pl.per_unit > 0) {
            hipLaunchKernelGGL(k_decode_balanced, dim3(static_cast<unsigned>(pl.units)), dim3(kThreads), 0, s,
                               pool->k, pool->v, static_cast<const uint16_t *>(d_q), static_cast<uint16_t *>(d_out),
                               d_seq_lens, d_block_table, bt_stride, reinterpret_cast<float *>(ws),
                               reinterpret_cast<float2 *>(ws + pl.off_ml),
                               reinterpret_cast<uint32_t *>(ws + pl.off_meta), next_tag(), pl.slots,
                               batch, pl.hkv, pl.group, pool->desc.num_pages, pl.scale_log2, pl.per_unit, pl.total,
                               pl.aligned ? 1 : 0);
            st = check_launch("k_decode_balanced");
        } else {
            hipLaunchKernelGGL(k_decode_split, dim3(static_cast<unsigned>(pl.units)), dim3(kThreads), 0, s,
                               pool->k, pool->v, static_cast<const uint16_t *>(d_q), static_cast<uint16_t *>(d_out),
                               d_seq_lens, d_block_table, bt_stride, reinterpret_cast<float *>(ws),
                               reinterpret_cast<float2 *>(ws + pl.off_ml),
                               reinterpret_cast<int32_t *>(ws + pl.off_meta), batch, pl.hkv, pl.group,
                               pool->desc.num_pages, pl.scale_log2, pl.chunk_pages);
            st = check_launch("k_decode_split");
        }
        if (st != MW_OK) return st;
    }
    st = timing_kernel_done(timing, s);
    if (st != MW_OK) return st;
    if (pl.per_unit == 0) {  // fixed chunks: the combine kernel
        st = decode_combine_launch(&a, pl, s);
        if (st != MW_OK) return st;
        st = timing_kernel_done(timing, s);
    }
    timing_end(timing);
    return st;
}

// Workspace of mw_decode_attn_noalloc: one array per device for the whole
// process, shared by every call on that device.  Host code never uses the
// array's name as an address (on the host it names a stand-in, not device
// memory): each device's address comes from hipGetSymbolAddress, taken once
// per device with that device current.
constexpr size_t kScratchBytes = size_t{16} << 20;
constexpr int kMaxDevices = 64;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices] = {};

mw_status scratch_for_stream(hipStream_t s, void **out, const char *who) {
    int dev = 0;
    if (s)
        MW_HIP_TRY(hipStreamGetDevice(s, &dev));
    else
        MW_HIP_TRY(hipGetDevice(&dev));
    if (dev < 0 || dev >= kMaxDevices) return fail(MW_ERR_UNSUPPORTED, "%s: device %d out of range", who, dev);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        int prev = 0;
        MW_HIP_TRY(hipGetDevice(&prev));
        if (prev != dev) MW_HIP_TRY(hipSetDevice(dev));
        void *ptr = nullptr;
        const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (prev != dev) (void)hipSetDevice(prev);
        if (e != hipSuccess || !ptr)
            return fail(MW_ERR_HIP, "%s: hipGetSymbolAddress(scratch) failed: %s", who, hipGetErrorString(e));
        g_scratch_ptr[dev] = ptr;
    }
    *out = g_scratch_ptr[dev];
    return MW_OK;
}

}  // namespace

extern "C" {

mw_status mw_decode_attn(const mw_kv_pool *pool, const mw_attn_shape *shape, int32_t batch,
                         const int32_t *h_seq_lens, const int32_t *d_seq_lens, const int32_t *d_block_table,
                         int32_t bt_stride, const void *d_q, void *d_out, void *d_workspace,
                         size_t workspace_bytes, int32_t chunk_pages, mw_stream stream, mw_timing *timing) {
    const char *who = "mw_decode_attn";
    if (!shape) return fail(MW_ERR_INVALID_ARG, "%s: bad arguments", who);
    const mw_decode_args a{pool,   *shape, batch,        h_seq_lens,      d_seq_lens, d_block_table,
                           bt_stride, d_q, d_out, d_workspace, workspace_bytes, chunk_pages};
    hipStream_t s = static_cast<hipStream_t>(stream);
    DecodePlan pl;
    mw_status st = decode_prepare(&a, stream_cus(s), &pl, who);
    if (st != MW_OK) return st;
    return decode_launch(a, pl, s, timing);
}

mw_status mw_decode_attn_noalloc(const mw_kv_pool *pool, const mw_attn_shape *shape, int32_t batch,
                                 const int32_t *h_seq_lens, const int32_t *d_seq_lens,
                                 const int32_t *d_block_table, int32_t bt_stride, const void *d_q,
                                 void *d_out, int32_t chunk_pages, mw_stream stream) {
    const char *who = "mw_decode_attn_noalloc";
    if (!shape) return fail(MW_ERR_INVALID_ARG, "%s: bad arguments", who);
    hipStream_t s = static_cast<hipStream_t>(stream);
    void *ws = nullptr;
    mw_status st = scratch_for_stream(s, &ws, who);
    if (st != MW_OK) return st;
    const mw_decode_args a{pool,      *shape, batch, h_seq_lens, d_seq_lens,    d_block_table,
                           bt_stride, d_q,    d_out, ws,         kScratchBytes, chunk_pages};
    // plan with an unbounded workspace first, so that a call too large for
    // the scratch array is reported as such
    mw_decode_args sized = a;
    sized.workspace_bytes = ~size_t{0};
    DecodePlan pl;
    st = decode_prepare(&sized, stream_cus(s), &pl, who);
    if (st != MW_OK) return st;
    if (pl.bytes > kScratchBytes)
        return fail(MW_ERR_UNSUPPORTED, "%s: the call needs %zu bytes of workspace, the static scratch holds %zu",
                    who, pl.bytes, kScratchBytes);
    return decode_launch(a, pl, s, nullptr);
}

}  // extern "C"
