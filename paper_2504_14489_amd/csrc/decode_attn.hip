// Decode attention: one query token per sequence over its paged context.
//
// Decode is memory-bound (paper Sec. 2.2: the decode phase is
// memory-intensive; Sec. 3.3, Table "tab:theory_cost": O(d^2 + (r+1) d)), so
// the design goal is streaming every K/V byte of the batch from HBM exactly
// once with enough bytes in flight, not arithmetic throughput.
//
// Work unit = (sequence b, kv head, chunk of CH consecutive pages).  The split
// depends only on the sequence lengths (never on page ids), so a result does
// not change when pages are renumbered.
//
// Per unit (4 waves, PPW = CH/4 pages per wave):
//   1. All K and V page rows of the wave are loaded up front (16-byte vector
//      loads; every lane has 16 loads of 16 B in flight per page pair).
//   2. Scores of the chunk's tokens against the G query heads of the kv head
//      come from one 16x16x32 bf16 MFMA per 32 dims: A = the page's K rows
//      [16 tokens x 32 dims] exactly as loaded from HBM, B = Q^T for the
//      group's heads (columns >= G are zero).  The MFMA is used only because
//      it reads K in its memory layout with no shuffles.
//   3. Max and sum over the chunk (per head) use cross-lane shuffles and a
//      4-entry LDS exchange; p = exp2(s*scale*log2e - m) stays in registers
//      and goes to LDS once for the value pass.
//   4. p*V on the vector ALU in fp32: each lane owns 8 dims of 4 tokens of a
//      page, so each V load instruction reads 4 whole 256-byte token rows.
//   5. Partials (m, l, unnormalised o) go to the workspace; a sequence with a
//      single chunk writes its normalised bf16 output directly.
// The combine kernel merges the chunks of each (sequence, kv head) with the
// log-sum-exp identity: M = max m_s, O = sum 2^(m_s-M) o_s / sum 2^(m_s-M) l_s.
#include "mw_internal.h"

using namespace mw;

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
constexpr float kLog2e = 1.4426950408889634f;

__device__ inline float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ inline float bf_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }
__device__ inline uint16_t to_bf16(float f) { return __builtin_bit_cast(uint16_t, static_cast<__bf16>(f)); }

__device__ inline int chunks_of(int L, int ch_pages, int bt_stride) {
    if (L <= 0) return 0;
    int np = (L + kPageSize - 1) / kPageSize;
    np = np < bt_stride ? np : bt_stride;
    return (np + ch_pages - 1) / ch_pages;
}

// Block-wide search for the sequence b and chunk c holding global chunk ci.
// s_loc = {b (or -1), c, first chunk index of b, chunks of b}.
__device__ void locate_chunk(const int32_t *__restrict__ seq_lens, int batch, int ch_pages,
                             int bt_stride, int ci, int *s_loc, int *s_wsum) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    if (threadIdx.x == 0) s_loc[0] = -1;
    __syncthreads();
    int running = 0;
    for (int base = 0; base < batch; base += kThreads) {
        const int b = base + threadIdx.x;
        const int n = b < batch ? chunks_of(seq_lens[b], ch_pages, bt_stride) : 0;
        int x = n;
        for (int off = 1; off < 64; off <<= 1) {
            const int y = __shfl_up(x, off);
            if (lane >= off) x += y;
        }
        if (lane == 63) s_wsum[wave] = x;
        __syncthreads();
        int wbase = 0, total = 0;
        for (int w = 0; w < kWaves; ++w) {
            const int v = s_wsum[w];
            total += v;
            if (w < wave) wbase += v;
        }
        const int incl = running + wbase + x, excl = incl - n;
        if (b < batch && ci >= excl && ci < incl) {
            s_loc[0] = b;
            s_loc[1] = ci - excl;
            s_loc[2] = excl;
            s_loc[3] = n;
        }
        running += total;
        __syncthreads();
    }
}

template <int GP, int PPW>
__global__ void __launch_bounds__(kThreads)
k_decode_split(const uint16_t *__restrict__ kpool, const uint16_t *__restrict__ vpool,
               const uint16_t *__restrict__ q, uint16_t *__restrict__ out,
               const int32_t *__restrict__ seq_lens, const int32_t *__restrict__ bt, int bt_stride,
               float *__restrict__ ws_o, float2 *__restrict__ ws_ml, int32_t *__restrict__ ws_cbase,
               int batch, int hkv, int group, int num_pages, float scale_log2) {
    constexpr int CH = kWaves * PPW;
    constexpr int kPBytes = CH * 16 * 16 * 4;            // p per [page][token][head]
    constexpr int kOBytes = kWaves * GP * kHeadDim * 4;  // per-wave partial o
    constexpr int kScratch = kPBytes > kOBytes ? kPBytes : kOBytes;
    __shared__ int s_loc[4];
    __shared__ int s_wsum[kWaves];
    __shared__ float s_red[kWaves][16];
    __shared__ float s_ml[2][16];
    __shared__ __attribute__((aligned(16))) float s_buf[kScratch / 4];

    const int u = blockIdx.x;
    const int kvh = u % hkv;
    locate_chunk(seq_lens, batch, CH, bt_stride, u / hkv, s_loc, s_wsum);
    const int b = s_loc[0];
    if (b < 0) return;  // more units launched than the device lengths give
    const int c = s_loc[1];
    const int nch = s_loc[3];

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int col = lane & 15, grp = lane >> 4;
    const int L = min(seq_lens[b], bt_stride * kPageSize);
    const int np_b = (L + kPageSize - 1) / kPageSize;
    const int p_begin = c * CH;
    const int p_end = min(p_begin + CH, np_b);
    const int32_t *btrow = bt + static_cast<size_t>(b) * bt_stride;
    const int hq = hkv * group;
    const uint4 zero4 = make_uint4(0, 0, 0, 0);

    // ---- issue every load of this wave: K (MFMA A layout) and V (row layout)
    uint4 kr[PPW][4], vr[PPW][4];
    bool pin[PPW];
#pragma unroll
    for (int i = 0; i < PPW; ++i) {
        const int p = p_begin + wave + kWaves * i;
        pin[i] = p < p_end;
        const int page = pin[i] ? btrow[p] : -1;
        const bool ok = page >= 0 && page < num_pages;
        const size_t base = (static_cast<size_t>(ok ? page : 0) * hkv + kvh) * (kPageSize * kHeadDim);
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
            kr[i][kb] = ok ? *reinterpret_cast<const uint4 *>(kpool + base + col * kHeadDim + 32 * kb + 8 * grp)
                           : zero4;
#pragma unroll
        for (int t4 = 0; t4 < 4; ++t4)
            vr[i][t4] = ok ? *reinterpret_cast<const uint4 *>(vpool + base + (4 * grp + t4) * kHeadDim + 8 * col)
                           : zero4;
    }

    // ---- Q^T operand: column `col` is query head kvh*group + col
    uint4 qop[4];
    {
        const bool hv = col < group;
        const uint16_t *qp = q + (static_cast<size_t>(b) * hq + kvh * group + (hv ? col : 0)) * kHeadDim + 8 * grp;
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) qop[kb] = hv ? *reinterpret_cast<const uint4 *>(qp + 32 * kb) : zero4;
    }

    // ---- scores: S^T[token][head], lane holds tokens 4*grp+r of head `col`
    f32x4 s[PPW];
    float mx = -INFINITY;
#pragma unroll
    for (int i = 0; i < PPW; ++i) {
        s[i] = f32x4{0.f, 0.f, 0.f, 0.f};
        if (pin[i]) {
#pragma unroll
            for (int kb = 0; kb < 4; ++kb)
                s[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, kr[i][kb]),
                                                               __builtin_bit_cast(bf16x8, qop[kb]), s[i], 0, 0, 0);
        }
        const int tok0 = (p_begin + wave + kWaves * i) * kPageSize + 4 * grp;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const float v = (pin[i] && tok0 + r < L) ? s[i][r] * scale_log2 : -INFINITY;
            s[i][r] = v;
            mx = fmaxf(mx, v);
        }
    }
    mx = fmaxf(mx, __shfl_xor(mx, 16));
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    if (grp == 0) s_red[wave][col] = mx;
    __syncthreads();
    const float m = fmaxf(fmaxf(s_red[0][col], s_red[1][col]), fmaxf(s_red[2][col], s_red[3][col]));

    float lsum = 0.f;
    float *s_p = s_buf;  // [CH][16 tokens][16 heads]
#pragma unroll
    for (int i = 0; i < PPW; ++i) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const float p = __builtin_amdgcn_exp2f(s[i][r] - m);
            lsum += p;
            s_p[((wave + kWaves * i) * 16 + 4 * grp + r) * 16 + col] = p;
        }
    }
    lsum += __shfl_xor(lsum, 16);
    lsum += __shfl_xor(lsum, 32);
    __syncthreads();  // everyone is past reading s_red for m
    if (grp == 0) s_red[wave][col] = lsum;
    __syncthreads();
    if (threadIdx.x < 16) {
        s_ml[0][col] = m;
        s_ml[1][col] = s_red[0][col] + s_red[1][col] + s_red[2][col] + s_red[3][col];
    }

    // ---- o = sum_t p[t][h] * v[t][:] on the vector ALU
    float acc[GP][8];
#pragma unroll
    for (int h = 0; h < GP; ++h)
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[h][e] = 0.f;
#pragma unroll
    for (int i = 0; i < PPW; ++i) {
        if (!pin[i]) continue;
#pragma unroll
        for (int t4 = 0; t4 < 4; ++t4) {
            const float *prow = s_p + ((wave + kWaves * i) * 16 + 4 * grp + t4) * 16;
            float pw[GP];
#pragma unroll
            for (int h = 0; h < GP; ++h) pw[h] = prow[h];
            const uint4 w = vr[i][t4];
            const float v8[8] = {bf_lo(w.x), bf_hi(w.x), bf_lo(w.y), bf_hi(w.y),
                                 bf_lo(w.z), bf_hi(w.z), bf_lo(w.w), bf_hi(w.w)};
#pragma unroll
            for (int h = 0; h < GP; ++h)
#pragma unroll
                for (int e = 0; e < 8; ++e) acc[h][e] = fmaf(pw[h], v8[e], acc[h][e]);
        }
    }
#pragma unroll
    for (int h = 0; h < GP; ++h)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            acc[h][e] += __shfl_xor(acc[h][e], 16);
            acc[h][e] += __shfl_xor(acc[h][e], 32);
        }
    __syncthreads();  // s_p is dead; reuse the buffer for per-wave partial o
    float *s_o = s_buf;  // [kWaves][GP][128]
    if (grp == 0) {
#pragma unroll
        for (int h = 0; h < GP; ++h)
#pragma unroll
            for (int e = 0; e < 8; ++e) s_o[(wave * GP + h) * kHeadDim + 8 * col + e] = acc[h][e];
    }
    __syncthreads();
    for (int idx = threadIdx.x; idx < group * kHeadDim; idx += kThreads) {
        const int h = idx / kHeadDim, d = idx % kHeadDim;
        float o = 0.f;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) o += s_o[(w * GP + h) * kHeadDim + d];
        if (nch == 1) {
            out[(static_cast<size_t>(b) * hq + kvh * group + h) * kHeadDim + d] = to_bf16(o / s_ml[1][h]);
        } else {
            ws_o[(static_cast<size_t>(u) * group + h) * kHeadDim + d] = o;
            if (d == 0) ws_ml[static_cast<size_t>(u) * group + h] = make_float2(s_ml[0][h], s_ml[1][h]);
        }
    }
    if (c == 0 && kvh == 0 && threadIdx.x == 0) ws_cbase[b] = s_loc[2];
}

__global__ void __launch_bounds__(kThreads)
k_decode_combine(uint16_t *__restrict__ out, const int32_t *__restrict__ seq_lens,
                 const float *__restrict__ ws_o, const float2 *__restrict__ ws_ml,
                 const int32_t *__restrict__ ws_cbase, int hkv, int group, int ch_pages, int bt_stride,
                 int total_chunks) {
    const int b = blockIdx.x / hkv, kvh = blockIdx.x % hkv;
    const int nch = chunks_of(seq_lens[b], ch_pages, bt_stride);
    if (nch <= 1) return;  // written by the split kernel
    const int cbase = ws_cbase[b];
    // lengths on the device that disagree with the host copy must not lead
    // outside the workspace
    if (cbase < 0 || cbase + nch > total_chunks) return;
    const int hq = hkv * group;
    for (int idx = threadIdx.x; idx < group * kHeadDim; idx += kThreads) {
        const int h = idx / kHeadDim, d = idx % kHeadDim;
        float M = -INFINITY;
        for (int sidx = 0; sidx < nch; ++sidx) {
            const float2 ml = ws_ml[(static_cast<size_t>(cbase + sidx) * hkv + kvh) * group + h];
            if (ml.y > 0.f) M = fmaxf(M, ml.x);
        }
        float lsum = 0.f, osum = 0.f;
        for (int sidx = 0; sidx < nch; ++sidx) {
            const size_t uu = (static_cast<size_t>(cbase + sidx) * hkv + kvh) * group + h;
            const float2 ml = ws_ml[uu];
            if (!(ml.y > 0.f)) continue;  // a chunk without keys contributes nothing
            const float w = __builtin_amdgcn_exp2f(ml.x - M);
            lsum += w * ml.y;
            osum += w * ws_o[uu * kHeadDim + d];
        }
        out[(static_cast<size_t>(b) * hq + kvh * group + h) * kHeadDim + d] = to_bf16(osum / lsum);
    }
}

struct Plan {
    int64_t units;
    size_t off_ml, off_cbase, bytes;
};

size_t align256(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }

mw_status plan_decode(const mw_attn_shape *shape, int32_t batch, const int32_t *h_seq_lens,
                      int32_t chunk_pages, int32_t bt_stride, Plan *plan, const char *who) {
    if (!shape || batch < 0 || (batch > 0 && !h_seq_lens))
        return fail(MW_ERR_INVALID_ARG, "%s: bad arguments", who);
    if (shape->head_dim != kHeadDim) return fail(MW_ERR_UNSUPPORTED, "%s: head_dim must be 128", who);
    if (shape->num_kv_heads < 1 || shape->num_q_heads < 1 || shape->num_q_heads % shape->num_kv_heads)
        return fail(MW_ERR_INVALID_ARG, "%s: num_q_heads must be a positive multiple of num_kv_heads", who);
    if (shape->num_q_heads / shape->num_kv_heads > 16)
        return fail(MW_ERR_UNSUPPORTED, "%s: at most 16 query heads per kv head", who);
    if (chunk_pages != 4 && chunk_pages != 8 && chunk_pages != 16)
        return fail(MW_ERR_UNSUPPORTED, "%s: chunk_pages must be 4, 8 or 16 (or 0)", who);
    int64_t chunks = 0;
    for (int32_t b = 0; b < batch; ++b) {
        const int32_t L = h_seq_lens[b];
        if (L < 1 || (bt_stride > 0 && static_cast<int64_t>(L) > static_cast<int64_t>(bt_stride) * kPageSize))
            return fail(MW_ERR_INVALID_ARG, "%s: sequence %d has length %d (table holds %d pages)", who, b,
                        L, bt_stride);
        chunks += ((L + kPageSize - 1) / kPageSize + chunk_pages - 1) / chunk_pages;
    }
    const int group = shape->num_q_heads / shape->num_kv_heads;
    plan->units = chunks * shape->num_kv_heads;
    const size_t o_bytes = align256(static_cast<size_t>(plan->units) * group * kHeadDim * 4);
    const size_t ml_bytes = align256(static_cast<size_t>(plan->units) * group * 8);
    plan->off_ml = o_bytes;
    plan->off_cbase = o_bytes + ml_bytes;
    plan->bytes = plan->off_cbase + align256(static_cast<size_t>(batch) * 4 + 4);
    return MW_OK;
}

template <int GP, int PPW>
void launch_split(dim3 grid, hipStream_t s, const mw_kv_pool *pool, const void *q, void *out,
                  const int32_t *seq_lens, const int32_t *bt, int bt_stride, char *ws, const Plan &pl,
                  int batch, int hkv, int group, float scale_log2) {
    hipLaunchKernelGGL((k_decode_split<GP, PPW>), grid, dim3(kThreads), 0, s, pool->k, pool->v,
                       static_cast<const uint16_t *>(q), static_cast<uint16_t *>(out), seq_lens, bt,
                       bt_stride, reinterpret_cast<float *>(ws), reinterpret_cast<float2 *>(ws + pl.off_ml),
                       reinterpret_cast<int32_t *>(ws + pl.off_cbase), batch, hkv, group,
                       pool->desc.num_pages, scale_log2);
}

template <int GP>
void launch_split_g(int ppw, dim3 grid, hipStream_t s, const mw_kv_pool *pool, const void *q, void *out,
                    const int32_t *seq_lens, const int32_t *bt, int bt_stride, char *ws, const Plan &pl,
                    int batch, int hkv, int group, float scale_log2) {
    switch (ppw) {
        case 1: launch_split<GP, 1>(grid, s, pool, q, out, seq_lens, bt, bt_stride, ws, pl, batch, hkv, group, scale_log2); break;
        case 2: launch_split<GP, 2>(grid, s, pool, q, out, seq_lens, bt, bt_stride, ws, pl, batch, hkv, group, scale_log2); break;
        default: launch_split<GP, 4>(grid, s, pool, q, out, seq_lens, bt, bt_stride, ws, pl, batch, hkv, group, scale_log2); break;
    }
}

}  // namespace

extern "C" {

mw_status mw_decode_workspace_size(const mw_attn_shape *shape, int32_t batch, const int32_t *h_seq_lens,
                                   int32_t chunk_pages, size_t *bytes) {
    if (!bytes) return fail(MW_ERR_INVALID_ARG, "mw_decode_workspace_size: bytes is NULL");
    Plan pl;
    mw_status st = plan_decode(shape, batch, h_seq_lens, chunk_pages ? chunk_pages : 16, 0, &pl,
                               "mw_decode_workspace_size");
    if (st != MW_OK) return st;
    *bytes = pl.bytes;
    return MW_OK;
}

mw_status mw_decode_attn(const mw_kv_pool *pool, const mw_attn_shape *shape, int32_t batch,
                         const int32_t *h_seq_lens, const int32_t *d_seq_lens, const int32_t *d_block_table,
                         int32_t bt_stride, const void *d_q, void *d_out, void *d_workspace,
                         size_t workspace_bytes, int32_t chunk_pages, mw_stream stream, mw_timing *timing) {
    const char *who = "mw_decode_attn";
    if (!pool || bt_stride < 1) return fail(MW_ERR_INVALID_ARG, "%s: bad pool or bt_stride", who);
    if (chunk_pages == 0) chunk_pages = 16;
    Plan pl;
    mw_status st = plan_decode(shape, batch, h_seq_lens, chunk_pages, bt_stride, &pl, who);
    if (st != MW_OK) return st;
    if (!(shape->scale > 0.f) || !(shape->scale < INFINITY))
        return fail(MW_ERR_INVALID_ARG, "%s: scale must be positive and finite", who);
    if (shape->num_kv_heads != pool->desc.num_kv_heads)
        return fail(MW_ERR_INVALID_ARG, "%s: num_kv_heads %d differs from the pool's %d", who,
                    shape->num_kv_heads, pool->desc.num_kv_heads);
    if (batch > 0 && (!d_seq_lens || !d_block_table || !d_q || !d_out || !d_workspace))
        return fail(MW_ERR_INVALID_ARG, "%s: NULL device pointer", who);
    if (batch > 0 && (!aligned16(d_q) || !aligned16(d_out) || !aligned16(d_workspace)))
        return fail(MW_ERR_INVALID_ARG, "%s: Q, O and workspace must be 16-byte aligned", who);
    if (workspace_bytes < pl.bytes)
        return fail(MW_ERR_INVALID_ARG, "%s: workspace of %zu bytes, %zu needed", who, workspace_bytes, pl.bytes);
    if (pl.units > 0x7fffffff) return fail(MW_ERR_UNSUPPORTED, "%s: too many work units", who);
    hipStream_t s = static_cast<hipStream_t>(stream);
    st = timing_begin(timing, s);
    if (st != MW_OK) return st;
    const int hkv = shape->num_kv_heads;
    const int group = shape->num_q_heads / hkv;
    const float scale_log2 = shape->scale * kLog2e;
    char *ws = static_cast<char *>(d_workspace);
    if (pl.units > 0) {
        const dim3 grid(static_cast<unsigned>(pl.units));
        const int ppw = chunk_pages / kWaves;
        if (group <= 1)
            launch_split_g<1>(ppw, grid, s, pool, d_q, d_out, d_seq_lens, d_block_table, bt_stride, ws, pl, batch, hkv, group, scale_log2);
        else if (group <= 2)
            launch_split_g<2>(ppw, grid, s, pool, d_q, d_out, d_seq_lens, d_block_table, bt_stride, ws, pl, batch, hkv, group, scale_log2);
        else if (group <= 4)
            launch_split_g<4>(ppw, grid, s, pool, d_q, d_out, d_seq_lens, d_block_table, bt_stride, ws, pl, batch, hkv, group, scale_log2);
        else if (group <= 8)
            launch_split_g<8>(ppw, grid, s, pool, d_q, d_out, d_seq_lens, d_block_table, bt_stride, ws, pl, batch, hkv, group, scale_log2);
        else
            launch_split_g<16>(ppw, grid, s, pool, d_q, d_out, d_seq_lens, d_block_table, bt_stride, ws, pl, batch, hkv, group, scale_log2);
        st = check_launch("k_decode_split");
        if (st != MW_OK) return st;
    }
    st = timing_kernel_done(timing, s);
    if (st != MW_OK) return st;
    if (batch > 0) {
        hipLaunchKernelGGL(k_decode_combine, dim3(static_cast<unsigned>(batch) * hkv), dim3(kThreads), 0, s,
                           static_cast<uint16_t *>(d_out), d_seq_lens, reinterpret_cast<const float *>(ws),
                           reinterpret_cast<const float2 *>(ws + pl.off_ml),
                           reinterpret_cast<const int32_t *>(ws + pl.off_cbase), hkv, group, chunk_pages,
                           bt_stride, static_cast<int>(pl.units / hkv));
        st = check_launch("k_decode_combine");
        if (st != MW_OK) return st;
    }
    st = timing_kernel_done(timing, s);
    timing_end(timing);
    return st;
}

}  // extern "C"
