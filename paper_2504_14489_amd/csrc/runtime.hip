// Host runtime: errors, timing events, the CU partition and the CU probe.
#include <hip/hip_ext.h>

#include <cstdarg>
#include <cstdio>
#include <cstring>

#include "mw_internal.h"

namespace mw {

static thread_local char g_last_error[512] = "";

mw_status fail(mw_status st, const char *fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_last_error, sizeof g_last_error, fmt, ap);
    va_end(ap);
    return st;
}

int stream_cus(hipStream_t s) {
    uint32_t mask[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    int n = 0;
    if (hipExtStreamGetCUMask(s, 8, mask) == hipSuccess)
        for (uint32_t m : mask) n += __builtin_popcount(m);
    if (n > 0) return n;
    (void)hipGetLastError();  // a failed query is not an error of the caller's work
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) == hipSuccess &&
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && cus > 0)
        return cus;
    (void)hipGetLastError();
    return 256;
}

mw_status check_launch(const char *what) {
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return fail(MW_ERR_HIP, "launch of %s failed: %s", what, hipGetErrorString(e));
    return MW_OK;
}

static mw_status timing_ensure_events(mw_timing *t) {
    if (t->created) return MW_OK;
    for (int i = 0; i < kMaxTimingEvents; ++i) MW_HIP_TRY(hipEventCreate(&t->ev[i]));
    t->created = true;
    return MW_OK;
}

mw_status timing_begin(mw_timing *t, hipStream_t s) {
    if (!t) return MW_OK;
    mw_status st = timing_ensure_events(t);
    if (st != MW_OK) return st;
    t->t0 = std::chrono::steady_clock::now();
    t->n_events = 0;
    MW_HIP_TRY(hipEventRecord(t->ev[0], s));
    t->n_events = 1;
    return MW_OK;
}

mw_status timing_kernel_done(mw_timing *t, hipStream_t s) {
    if (!t) return MW_OK;
    if (t->n_events >= kMaxTimingEvents) return fail(MW_ERR_INVALID_ARG, "too many timed kernels");
    MW_HIP_TRY(hipEventRecord(t->ev[t->n_events], s));
    ++t->n_events;
    return MW_OK;
}

void timing_end(mw_timing *t) {
    if (!t) return;
    t->host_ms =
        std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t->t0).count();
}

}  // namespace mw

using namespace mw;

extern "C" {

const char *mw_last_error(void) { return g_last_error; }

int32_t mw_version(void) { return 2; }

mw_status mw_sync(mw_stream stream) {
    MW_HIP_TRY(hipStreamSynchronize(static_cast<hipStream_t>(stream)));
    MW_HIP_TRY(hipGetLastError());
    return MW_OK;
}

// ---------------------------------------------------------------- timing --
mw_status mw_timing_create(mw_timing **out) {
    if (!out) return fail(MW_ERR_INVALID_ARG, "mw_timing_create: out is NULL");
    mw_timing *t = new (std::nothrow) mw_timing();
    if (!t) return fail(MW_ERR_INVALID_ARG, "mw_timing_create: out of host memory");
    t->n_events = 0;
    t->created = false;
    t->host_ms = 0.0;
    *out = t;
    return MW_OK;
}

mw_status mw_timing_destroy(mw_timing *t) {
    if (!t) return MW_OK;
    if (t->created)
        for (int i = 0; i < kMaxTimingEvents; ++i) (void)hipEventDestroy(t->ev[i]);
    delete t;
    return MW_OK;
}

mw_status mw_timing_mark(mw_timing *t, mw_stream stream) {
    if (!t) return fail(MW_ERR_INVALID_ARG, "mw_timing_mark: NULL timing");
    mw_status st = timing_begin(t, static_cast<hipStream_t>(stream));
    timing_end(t);
    return st;
}

static mw_status timing_ready(mw_timing *t, const char *who) {
    if (!t) return fail(MW_ERR_INVALID_ARG, "%s: NULL timing", who);
    if (!t->created || t->n_events < 1) return fail(MW_ERR_NOT_READY, "%s: nothing recorded", who);
    MW_HIP_TRY(hipEventSynchronize(t->ev[t->n_events - 1]));
    return MW_OK;
}

mw_status mw_timing_elapsed(mw_timing *t, float *gpu_ms, float *host_launch_ms) {
    mw_status st = timing_ready(t, "mw_timing_elapsed");
    if (st != MW_OK) return st;
    if (gpu_ms) {
        *gpu_ms = 0.f;
        if (t->n_events > 1) MW_HIP_TRY(hipEventElapsedTime(gpu_ms, t->ev[0], t->ev[t->n_events - 1]));
    }
    if (host_launch_ms) *host_launch_ms = static_cast<float>(t->host_ms);
    return MW_OK;
}

mw_status mw_timing_kernels(mw_timing *t, int32_t *n_kernels) {
    if (!t || !n_kernels) return fail(MW_ERR_INVALID_ARG, "mw_timing_kernels: NULL argument");
    *n_kernels = t->n_events > 0 ? t->n_events - 1 : 0;
    return MW_OK;
}

mw_status mw_timing_kernel_ms(mw_timing *t, int32_t k, float *ms) {
    mw_status st = timing_ready(t, "mw_timing_kernel_ms");
    if (st != MW_OK) return st;
    if (!ms || k < 0 || k + 1 >= t->n_events)
        return fail(MW_ERR_INVALID_ARG, "mw_timing_kernel_ms: kernel %d not recorded", k);
    MW_HIP_TRY(hipEventElapsedTime(ms, t->ev[k], t->ev[k + 1]));
    return MW_OK;
}

mw_status mw_timing_offsets(mw_timing *t, mw_timing *ref, float *start_ms, float *stop_ms) {
    mw_status st = timing_ready(t, "mw_timing_offsets");
    if (st != MW_OK) return st;
    st = timing_ready(ref, "mw_timing_offsets(ref)");
    if (st != MW_OK) return st;
    if (start_ms) MW_HIP_TRY(hipEventElapsedTime(start_ms, ref->ev[0], t->ev[0]));
    if (stop_ms) MW_HIP_TRY(hipEventElapsedTime(stop_ms, ref->ev[0], t->ev[t->n_events - 1]));
    return MW_OK;
}

// ------------------------------------------------------------- partition --
static mw_status make_stream(int device, const uint32_t *mask, int n_words, hipStream_t *s) {
    int prev = 0;
    MW_HIP_TRY(hipGetDevice(&prev));
    MW_HIP_TRY(hipSetDevice(device));
    hipError_t e = hipExtStreamCreateWithCUMask(s, static_cast<uint32_t>(n_words), mask);
    (void)hipSetDevice(prev);
    if (e != hipSuccess)
        return fail(MW_ERR_HIP, "hipExtStreamCreateWithCUMask failed: %s", hipGetErrorString(e));
    return MW_OK;
}

mw_status mw_partition_create_masks(int32_t device, const uint32_t *prefill_mask,
                                    const uint32_t *decode_mask, int32_t n_words,
                                    mw_partition **out) {
    if (!prefill_mask || !decode_mask || !out || n_words < 1 || n_words > 8)
        return fail(MW_ERR_INVALID_ARG, "mw_partition_create_masks: bad arguments");
    int n_dev = 0;
    MW_HIP_TRY(hipGetDeviceCount(&n_dev));
    if (device < 0 || device >= n_dev)
        return fail(MW_ERR_INVALID_ARG, "mw_partition_create_masks: no device %d", device);
    bool any_p = false, any_d = false;
    for (int w = 0; w < n_words; ++w) {
        if (prefill_mask[w] & decode_mask[w])
            return fail(MW_ERR_INVALID_ARG, "mw_partition_create_masks: masks overlap in word %d", w);
        any_p |= prefill_mask[w] != 0;
        any_d |= decode_mask[w] != 0;
    }
    if (!any_p || !any_d) return fail(MW_ERR_INVALID_ARG, "mw_partition_create_masks: empty mask");
    mw_partition *p = new (std::nothrow) mw_partition();
    if (!p) return fail(MW_ERR_INVALID_ARG, "mw_partition_create_masks: out of host memory");
    p->device = device;
    std::memset(p->prefill_mask, 0, sizeof p->prefill_mask);
    std::memset(p->decode_mask, 0, sizeof p->decode_mask);
    std::memcpy(p->prefill_mask, prefill_mask, sizeof(uint32_t) * n_words);
    std::memcpy(p->decode_mask, decode_mask, sizeof(uint32_t) * n_words);
    mw_status st = make_stream(device, p->prefill_mask, n_words, &p->prefill);
    if (st != MW_OK) {
        delete p;
        return st;
    }
    st = make_stream(device, p->decode_mask, n_words, &p->decode);
    if (st != MW_OK) {
        (void)hipStreamDestroy(p->prefill);
        delete p;
        return st;
    }
    *out = p;
    return MW_OK;
}

// The runtime numbers the CUs of a multi-XCD device round-robin over the
// XCDs (CU c sits on XCD c % n_xcd), so the first 8k mask bits select k CUs on
// each of the 8 XCDs.  Prefill takes bits [0, prefill_cus), decode the next
// decode_cus bits.
mw_status mw_partition_create(int32_t device, int32_t prefill_cus, int32_t decode_cus,
                              mw_partition **out) {
    int n_dev = 0;
    MW_HIP_TRY(hipGetDeviceCount(&n_dev));
    if (device < 0 || device >= n_dev)
        return fail(MW_ERR_INVALID_ARG, "mw_partition_create: no device %d", device);
    int n_cu = 0;
    MW_HIP_TRY(hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, device));
    if (prefill_cus < 8 || decode_cus < 8 || prefill_cus % 8 || decode_cus % 8 ||
        prefill_cus + decode_cus > n_cu || n_cu > 256)
        return fail(MW_ERR_INVALID_ARG,
                    "mw_partition_create: CU counts %d/%d must be multiples of 8, >= 8 each, "
                    "summing to at most %d",
                    prefill_cus, decode_cus, n_cu);
    uint32_t pm[8] = {0}, dm[8] = {0};
    for (int c = 0; c < prefill_cus; ++c) pm[c / 32] |= 1u << (c % 32);
    for (int c = prefill_cus; c < prefill_cus + decode_cus; ++c) dm[c / 32] |= 1u << (c % 32);
    return mw_partition_create_masks(device, pm, dm, (n_cu + 31) / 32, out);
}

mw_status mw_partition_streams(const mw_partition *part, mw_stream *prefill, mw_stream *decode) {
    if (!part) return fail(MW_ERR_INVALID_ARG, "mw_partition_streams: NULL partition");
    if (prefill) *prefill = part->prefill;
    if (decode) *decode = part->decode;
    return MW_OK;
}

mw_status mw_partition_masks(const mw_partition *part, uint32_t *prefill_mask,
                             uint32_t *decode_mask) {
    if (!part) return fail(MW_ERR_INVALID_ARG, "mw_partition_masks: NULL partition");
    if (prefill_mask) std::memcpy(prefill_mask, part->prefill_mask, sizeof part->prefill_mask);
    if (decode_mask) std::memcpy(decode_mask, part->decode_mask, sizeof part->decode_mask);
    return MW_OK;
}

mw_status mw_partition_destroy(mw_partition *part) {
    if (!part) return MW_OK;
    hipError_t e1 = hipStreamSynchronize(part->prefill);
    hipError_t e2 = hipStreamSynchronize(part->decode);
    (void)hipStreamDestroy(part->prefill);
    (void)hipStreamDestroy(part->decode);
    delete part;
    if (e1 != hipSuccess || e2 != hipSuccess)
        return fail(MW_ERR_HIP, "mw_partition_destroy: %s",
                    hipGetErrorString(e1 != hipSuccess ? e1 : e2));
    return MW_OK;
}

}  // extern "C"

// --------------------------------------------------------------- probe ----
// hwreg ids: HW_ID (4) and XCC_ID (20); s_getreg immediate = (size-1)<<11 | offset<<6 | id
__global__ void __launch_bounds__(64) k_cu_probe(uint32_t *out, int spin_cycles) {
    const uint32_t hw = __builtin_amdgcn_s_getreg((31 << 11) | (0 << 6) | 4);
    const uint32_t xcc = __builtin_amdgcn_s_getreg((15 << 11) | (0 << 6) | 20);
    const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
    const uint64_t c0 = __builtin_readcyclecounter();
    while (__builtin_readcyclecounter() - c0 < static_cast<uint64_t>(spin_cycles)) {
        __builtin_amdgcn_s_sleep(1);
    }
    const uint64_t t1 = __builtin_amdgcn_s_memrealtime();
    if (threadIdx.x == 0) {
        uint32_t *o = out + 4 * static_cast<size_t>(blockIdx.x);
        o[0] = xcc;
        o[1] = hw;
        o[2] = static_cast<uint32_t>(t0);
        o[3] = static_cast<uint32_t>(t1);
    }
}

extern "C" mw_status mw_cu_probe(int32_t n_blocks, int32_t spin_cycles, uint32_t *d_out,
                                 mw_stream stream, mw_timing *timing) {
    if (n_blocks < 1 || n_blocks > (1 << 20) || spin_cycles < 0 || spin_cycles > (1 << 26) || !d_out)
        return fail(MW_ERR_INVALID_ARG, "mw_cu_probe: bad arguments");
    hipStream_t s = static_cast<hipStream_t>(stream);
    mw_status st = timing_begin(timing, s);
    if (st != MW_OK) return st;
    hipLaunchKernelGGL(k_cu_probe, dim3(n_blocks), dim3(64), 0, s, d_out, spin_cycles);
    st = check_launch("k_cu_probe");
    if (st != MW_OK) return st;
    st = timing_kernel_done(timing, s);
    timing_end(timing);
    return st;
}

// ------------------------------------------------------- stream read ------
// Reads `bytes` (a multiple of 16) once with 16-byte loads, grid-stride, 8
// loads in flight per thread; each block folds what it read into one word of
// d_sink[block] so the loads cannot be dropped.
__global__ void __launch_bounds__(256) k_stream_read(const uint4 *__restrict__ src, size_t n_vec,
                                                     uint32_t *__restrict__ sink) {
    const size_t stride = static_cast<size_t>(gridDim.x) * blockDim.x;
    size_t i = static_cast<size_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    uint32_t acc = 0;
    for (; i + 7 * stride < n_vec; i += 8 * stride) {
        uint4 v[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) v[j] = src[i + j * stride];
#pragma unroll
        for (int j = 0; j < 8; ++j) acc ^= v[j].x ^ v[j].y ^ v[j].z ^ v[j].w;
    }
    for (; i < n_vec; i += stride) {
        const uint4 v = src[i];
        acc ^= v.x ^ v.y ^ v.z ^ v.w;
    }
    __shared__ uint32_t red[256];
    red[threadIdx.x] = acc;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t a = 0;
        for (int t = 0; t < 256; ++t) a ^= red[t];
        sink[blockIdx.x] = a;
    }
}

extern "C" mw_status mw_stream_read(const void *d_src, size_t bytes, uint32_t *d_sink, int32_t n_blocks,
                                    mw_stream stream, mw_timing *timing) {
    if (!d_src || !d_sink || bytes % 16 || !aligned16(d_src) || n_blocks < 1 || n_blocks > (1 << 20))
        return fail(MW_ERR_INVALID_ARG, "mw_stream_read: bad arguments");
    hipStream_t s = static_cast<hipStream_t>(stream);
    mw_status st = timing_begin(timing, s);
    if (st != MW_OK) return st;
    hipLaunchKernelGGL(k_stream_read, dim3(n_blocks), dim3(256), 0, s, static_cast<const uint4 *>(d_src),
                       bytes / 16, d_sink);
    st = check_launch("k_stream_read");
    if (st != MW_OK) return st;
    st = timing_kernel_done(timing, s);
    timing_end(timing);
    return st;
}

// ----------------------------------------------------------- cache flush ----
// Reads the buffer past its first 16 KiB once with 16-byte loads: run between
// isolated timed calls, it evicts what the previous call left in the L2 of
// every XCD the stream runs on and in the memory-side Infinity Cache, leaving
// only clean lines (a flush by writing would leave dirty lines whose
// write-back the next, timed, kernel would pay for).  Each work-group folds
// what it read into one word of the buffer's first 8 KiB.
constexpr int kFlushBlocks = 2048;
constexpr size_t kFlushSkip = 16384;

__global__ void __launch_bounds__(256) k_cache_flush(uint4 *__restrict__ buf, size_t n_vec) {
    const uint4 *src = buf + kFlushSkip / 16;
    const size_t stride = static_cast<size_t>(gridDim.x) * blockDim.x;
    uint32_t acc = 0;
    size_t i = static_cast<size_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    for (; i + 3 * stride < n_vec; i += 4 * stride) {
        uint4 v[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) v[j] = src[i + j * stride];
#pragma unroll
        for (int j = 0; j < 4; ++j) acc ^= v[j].x ^ v[j].y ^ v[j].z ^ v[j].w;
    }
    for (; i < n_vec; i += stride) {
        const uint4 v = src[i];
        acc ^= v.x ^ v.y ^ v.z ^ v.w;
    }
    acc = __reduce_or_sync(~0ull, acc);
    if (threadIdx.x == 0) reinterpret_cast<uint32_t *>(buf)[blockIdx.x] = acc;
}

extern "C" mw_status mw_cache_flush(void *d_buf, size_t bytes, mw_stream stream) {
    if (!d_buf || bytes % 16 || !aligned16(d_buf) || bytes <= kFlushSkip)
        return fail(MW_ERR_INVALID_ARG, "mw_cache_flush: bad arguments");
    hipStream_t s = static_cast<hipStream_t>(stream);
    hipLaunchKernelGGL(k_cache_flush, dim3(kFlushBlocks), dim3(256), 0, s, static_cast<uint4 *>(d_buf),
                       (bytes - kFlushSkip) / 16);
    return check_launch("k_cache_flush");
}

// ------------------------------------------------------------ MFMA peak -----
// Each wave issues `iters` rounds of four independent bf16 32x32x16 MFMAs
// (32768 flop each) from registers: the matrix-core throughput the CUs of a
// stream sustain at the clock the chip holds under that load.  The result is
// folded into d_sink[block] so the products cannot be dropped.
typedef __bf16 mp_bf16x8 __attribute__((ext_vector_type(8)));
typedef float mp_f32x16 __attribute__((ext_vector_type(16)));

__global__ void __launch_bounds__(256) k_mfma_peak(float *__restrict__ sink, int iters) {
    const float x = 1e-3f * static_cast<float>((threadIdx.x & 7) + 1);
    mp_bf16x8 a, b;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        a[i] = static_cast<__bf16>(x);
        b[i] = static_cast<__bf16>(x * 0.5f);
    }
    mp_f32x16 acc[4];
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[j][i] = 0.f;
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[j], 0, 0, 0);
    }
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int i = 0; i < 16; ++i) s += acc[j][i];
    if (threadIdx.x == 0) sink[blockIdx.x] = s;
}

extern "C" mw_status mw_mfma_peak(int32_t n_blocks, int32_t iters, float *d_sink, mw_stream stream,
                                  mw_timing *timing, double *flop) {
    if (n_blocks < 1 || n_blocks > (1 << 20) || iters < 1 || iters > (1 << 24) || !d_sink)
        return fail(MW_ERR_INVALID_ARG, "mw_mfma_peak: bad arguments");
    hipStream_t s = static_cast<hipStream_t>(stream);
    mw_status st = timing_begin(timing, s);
    if (st != MW_OK) return st;
    hipLaunchKernelGGL(k_mfma_peak, dim3(n_blocks), dim3(256), 0, s, d_sink, iters);
    st = check_launch("k_mfma_peak");
    if (st != MW_OK) return st;
    st = timing_kernel_done(timing, s);
    timing_end(timing);
    if (flop) *flop = static_cast<double>(n_blocks) * 4 * static_cast<double>(iters) * 4 * 32768.0;
    return st;
}

// ------------------------------------------------------------ trace mark ----
// An empty kernel of `id` one-wave work-groups: a kernel trace shows it as
// k_trace_mark with grid size 64 * id, which lets a trace reader find the
// points where a program marked itself (the start and end of a timed region).
__global__ void __launch_bounds__(64) k_trace_mark() {}

extern "C" mw_status mw_trace_mark(int32_t id, mw_stream stream) {
    if (id < 1 || id > (1 << 16)) return fail(MW_ERR_INVALID_ARG, "mw_trace_mark: id must be in [1, 65536]");
    hipLaunchKernelGGL(k_trace_mark, dim3(id), dim3(64), 0, static_cast<hipStream_t>(stream));
    return check_launch("k_trace_mark");
}
