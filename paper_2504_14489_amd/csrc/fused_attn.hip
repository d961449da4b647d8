// One launch covering a prefill batch and a decode batch: the fused
// comparator for spatial multiplexing.  Chunked-prefill systems run both
// attentions in one kernel over the whole GPU (paper Sec. 4.1, the SGLang
// chunked-prefill baseline with its fused prefill + decode attention); here
// that is a kernel whose work-groups are either a prefill work-group (the
// body of the prefill kernel) or two decode work units (the body of the
// decode split kernel on each half of the 8 waves), followed by the decode
// combine kernel.  Prefill work-groups and decode pairs are interleaved in
// dispatch order in proportion to their counts, so every CU runs a mix of
// both while the launch lasts; no CU is set aside for either phase.
#include "decode_block.h"
#include "prefill_block.h"

using namespace mw;

namespace {

constexpr int kThreadsFused = 512;
static_assert(pf::kThreads == kThreadsFused && 2 * dk::kThreads == kThreadsFused,
              "a fused work-group is one prefill work-group or two decode units");
// LDS: prefill K tiles | V tiles | block-table copy, or per decode half its V
// buffers and (m, l) slots
constexpr int kPrefillK = 0;
constexpr int kPrefillV = 2 * pf::TILE * 2;
constexpr int kPrefillBt = 4 * pf::TILE * 2;
constexpr int kPrefillBytes = kPrefillBt + pf::kBtCache * 4;
constexpr int kDecodeV = dk::kWaves * dk::kWaveBufElems * 2;
constexpr int kDecodeHalf = kDecodeV + 2 * dk::kWaves * 16 * 4;
constexpr int kLdsBytes = kPrefillBytes > 2 * kDecodeHalf ? kPrefillBytes : 2 * kDecodeHalf;
static_assert(kDecodeHalf % 16 == 0, "decode LDS halves stay 16-byte aligned");

template <bool kTableInLds>
__global__ void __launch_bounds__(kThreadsFused, 1)
k_fused_attn(const uint16_t *__restrict__ kpool, const uint16_t *__restrict__ vpool, int num_pages, int hkv,
             // prefill
             const uint16_t *__restrict__ pq, uint16_t *__restrict__ pout, const int32_t *__restrict__ qo_indptr,
             const int32_t *__restrict__ prefix_lens, const int32_t *__restrict__ pbt, int pbt_stride, int pgroup,
             float pscale_log2, int paired, int n_hgroups, int gx, int64_t n_pre,
             // decode
             const uint16_t *__restrict__ dq, uint16_t *__restrict__ dout, const int32_t *__restrict__ seq_lens,
             const int32_t *__restrict__ dbt, int dbt_stride, float *__restrict__ ws_o, float2 *__restrict__ ws_ml,
             int32_t *__restrict__ ws_cbase, int dbatch, int dgroup, float dscale_log2, int ch_pages,
             int64_t n_dec) {
    __shared__ __attribute__((aligned(1024))) char lds[kLdsBytes];
    // block i is prefill work-group floor(i P / T) when that index steps up at
    // i, else decode pair i - floor((i + 1) P / T)  (P + D = T blocks)
    const int64_t i = blockIdx.x, total = n_pre + n_dec;
    const int64_t p_lo = i * n_pre / total, p_hi = (i + 1) * n_pre / total;
    if (p_hi > p_lo) {
        const int x = static_cast<int>(p_lo % gx), b = static_cast<int>(p_lo / gx);
        pf::prefill_block<kTableInLds, 8>(kpool, vpool, pq, pout, qo_indptr, prefix_lens, pbt, pbt_stride, hkv, pgroup,
                                       num_pages, pscale_log2, paired, n_hgroups, x, b,
                                       reinterpret_cast<uint16_t *>(lds + kPrefillK),
                                       reinterpret_cast<uint16_t *>(lds + kPrefillV),
                                       reinterpret_cast<int32_t *>(lds + kPrefillBt));
    } else {
        const int64_t pair = i - p_hi;
        const int half = threadIdx.x >> 8;
        char *mine = lds + half * kDecodeHalf;
        float(*s_m)[16] = reinterpret_cast<float(*)[16]>(mine + kDecodeV);
        float(*s_l)[16] = reinterpret_cast<float(*)[16]>(mine + kDecodeV + dk::kWaves * 16 * 4);
        dk::decode_unit<true>(kpool, vpool, dq, dout, seq_lens, dbt, dbt_stride, ws_o, ws_ml, ws_cbase, dbatch, hkv,
                              dgroup, num_pages, dscale_log2, ch_pages, static_cast<int>(2 * pair + half),
                              threadIdx.x & 255, reinterpret_cast<uint16_t *>(mine), s_m, s_l);
    }
}

}  // namespace

extern "C" mw_status mw_fused_attn(const mw_prefill_args *pre, const mw_decode_args *dec, mw_stream stream,
                                   mw_timing *timing) {
    const char *who = "mw_fused_attn";
    if (!pre || !dec) return fail(MW_ERR_INVALID_ARG, "%s: NULL argument", who);
    if (pre->pool != dec->pool) return fail(MW_ERR_INVALID_ARG, "%s: prefill and decode must share one pool", who);
    hipStream_t s = static_cast<hipStream_t>(stream);
    PrefillPlan pp;
    mw_status st = prefill_prepare(pre, stream_cus(s), false, &pp, who);  // 8-wave work-groups only
    if (st != MW_OK) return st;
    DecodePlan dp;
    st = decode_prepare(dec, 0, &dp, who);  // fixed chunks: a fused work-group's barriers are uniform
    if (st != MW_OK) return st;
    const int64_t n_pre = pp.gx * pp.batch, n_dec = (dp.units + 1) / 2;
    if (n_pre + n_dec > 0x7fffffff) return fail(MW_ERR_UNSUPPORTED, "%s: grid too large", who);
    st = timing_begin(timing, s);
    if (st != MW_OK) return st;
    if (n_pre + n_dec > 0) {
        const mw_kv_pool *pool = pre->pool;
        char *ws = static_cast<char *>(dec->d_workspace);
        auto kernel = pp.table_in_lds ? k_fused_attn<true> : k_fused_attn<false>;
        hipLaunchKernelGGL(kernel, dim3(static_cast<unsigned>(n_pre + n_dec)), dim3(kThreadsFused), 0, s, pool->k,
                           pool->v, pool->desc.num_pages, pp.hkv, static_cast<const uint16_t *>(pre->d_q),
                           static_cast<uint16_t *>(pre->d_out), pre->d_qo_indptr, pre->d_prefix_lens,
                           pre->d_block_table, pre->bt_stride, pp.group, pp.scale_log2, pp.paired, pp.n_hgroups,
                           static_cast<int>(pp.gx > 0 ? pp.gx : 1), n_pre, static_cast<const uint16_t *>(dec->d_q),
                           static_cast<uint16_t *>(dec->d_out), dec->d_seq_lens, dec->d_block_table, dec->bt_stride,
                           reinterpret_cast<float *>(ws), reinterpret_cast<float2 *>(ws + dp.off_ml),
                           reinterpret_cast<int32_t *>(ws + dp.off_meta), dec->batch, dp.group, dp.scale_log2,
                           dp.chunk_pages, n_dec);
        st = check_launch("k_fused_attn");
        if (st != MW_OK) return st;
    }
    st = timing_kernel_done(timing, s);
    if (st != MW_OK) return st;
    st = decode_combine_launch(dec, dp, s);
    if (st != MW_OK) return st;
    st = timing_kernel_done(timing, s);
    timing_end(timing);
    return st;
}
