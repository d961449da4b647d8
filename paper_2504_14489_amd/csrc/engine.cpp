// Bubble-less multiplex engine (paper Sec. 3.2): a group of CU partitions
// created once, and a host loop that feeds decode iterations and prefill
// layers to their streams, either blocking on every decode iteration (the
// naive integration the paper starts from) or polling events (its
// query-based synchronization) with layer-wise prefill launches and a switch
// of the remaining prefill layers to the whole device when decode ends.
#include <hip/hip_ext.h>

#include <algorithm>
#include <chrono>
#include <cstring>
#include <new>
#include <vector>

#include "mw_internal.h"

using namespace mw;

struct mw_engine {
    int device;
    int n;
    int32_t prefill_cus[16], decode_cus[16];
    hipStream_t prefill[16], decode[16];
    hipStream_t whole;
    int64_t mem_bytes;
    double create_ms;
    // the last run's calls: (start ms, end ms, 1 if on the whole device)
    std::vector<double> timeline[2];
    // captured decode iterations, one per (partition, decode arguments,
    // lengths, layer count)
    struct Graph {
        int config, layers;
        std::vector<unsigned char> key;
        hipGraph_t graph;
        hipGraphExec_t exec;
        int64_t bytes;
        double capture_ms;
    };
    std::vector<Graph> graphs;
};

namespace {

using clk = std::chrono::steady_clock;

double ms_since(clk::time_point t0) { return std::chrono::duration<double, std::milli>(clk::now() - t0).count(); }

mw_status masked_stream(int n_words, const uint32_t *mask, hipStream_t *s) {
    const hipError_t e = hipExtStreamCreateWithCUMask(s, static_cast<uint32_t>(n_words), mask);
    if (e != hipSuccess) return fail(MW_ERR_HIP, "hipExtStreamCreateWithCUMask failed: %s", hipGetErrorString(e));
    return MW_OK;
}

void destroy_graphs(mw_engine *e) {
    for (mw_engine::Graph &g : e->graphs) {
        (void)hipGraphExecDestroy(g.exec);
        (void)hipGraphDestroy(g.graph);
    }
    e->graphs.clear();
}

void destroy_streams(mw_engine *e) {
    for (int i = 0; i < e->n; ++i) {
        if (e->prefill[i]) (void)hipStreamDestroy(e->prefill[i]);
        if (e->decode[i]) (void)hipStreamDestroy(e->decode[i]);
    }
    if (e->whole) (void)hipStreamDestroy(e->whole);
}

// A pair of events around one launch on one stream.
struct Span {
    hipEvent_t start, end;
};

struct EventPool {
    std::vector<hipEvent_t> all;
    size_t used = 0;
    mw_status get(hipEvent_t *ev) {
        if (used == all.size()) {
            hipEvent_t e;
            MW_HIP_TRY(hipEventCreate(&e));
            all.push_back(e);
        }
        *ev = all[used++];
        return MW_OK;
    }
    ~EventPool() {
        for (hipEvent_t e : all) (void)hipEventDestroy(e);
    }
};

mw_status check_args(const mw_engine *eng, const mw_decode_args *dec, const mw_prefill_args *pre,
                     const mw_engine_plan *pl) {
    if (!eng || !dec || !pre || !pl) return fail(MW_ERR_INVALID_ARG, "mw_engine_run: NULL argument");
    if (pl->config < 0 || pl->config >= eng->n)
        return fail(MW_ERR_INVALID_ARG, "mw_engine_run: config %d outside [0, %d)", pl->config, eng->n);
    if (pl->decode_iters < 1 || pl->decode_layers < 1 || pl->prefill_layers < 1 || pl->layers_per_launch < 1)
        return fail(MW_ERR_INVALID_ARG, "mw_engine_run: iteration and layer counts must be >= 1");
    if (pl->policy != MW_ENGINE_BLOCKING && pl->policy != MW_ENGINE_POLLED)
        return fail(MW_ERR_INVALID_ARG, "mw_engine_run: unknown policy %d", pl->policy);
    if (pl->decode_graph != 0 && pl->decode_graph != 1)
        return fail(MW_ERR_INVALID_ARG, "mw_engine_run: decode_graph must be 0 or 1");
    if (pl->decode_graph && dec->batch > (1 << 20))
        return fail(MW_ERR_INVALID_ARG, "mw_engine_run: decode batch too large");
    return MW_OK;
}

// Cache key of a decode graph: the decode arguments field by field (never the
// struct's bytes, whose padding a caller need not initialise), the lengths'
// values rather than where the host keeps them, and the layer count.
std::vector<unsigned char> graph_key(const mw_decode_args *dec, int layers) {
    std::vector<unsigned char> k;
    auto put = [&k](const void *p, size_t n) {
        const unsigned char *b = static_cast<const unsigned char *>(p);
        k.insert(k.end(), b, b + n);
    };
    const void *ptrs[6] = {dec->pool, dec->d_seq_lens, dec->d_block_table, dec->d_q, dec->d_out, dec->d_workspace};
    put(ptrs, sizeof ptrs);
    const int32_t ints[6] = {dec->shape.num_q_heads, dec->shape.num_kv_heads, dec->shape.head_dim, dec->batch,
                             dec->bt_stride, dec->chunk_pages};
    put(ints, sizeof ints);
    put(&dec->shape.scale, sizeof dec->shape.scale);
    put(&dec->workspace_bytes, sizeof dec->workspace_bytes);
    put(&layers, sizeof layers);
    if (dec->batch > 0 && dec->h_seq_lens) put(dec->h_seq_lens, sizeof(int32_t) * static_cast<size_t>(dec->batch));
    return k;
}

}  // namespace

extern "C" {

mw_status mw_engine_create(int32_t device, const int32_t *prefill_cus, int32_t n, mw_engine **out) {
    if (!prefill_cus || !out || n < 1 || n > 16) return fail(MW_ERR_INVALID_ARG, "mw_engine_create: bad arguments");
    int n_dev = 0;
    MW_HIP_TRY(hipGetDeviceCount(&n_dev));
    if (device < 0 || device >= n_dev) return fail(MW_ERR_INVALID_ARG, "mw_engine_create: no device %d", device);
    int n_cu = 0;
    MW_HIP_TRY(hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, device));
    if (n_cu > 256) return fail(MW_ERR_UNSUPPORTED, "mw_engine_create: %d CUs (at most 256)", n_cu);
    for (int i = 0; i < n; ++i)
        if (prefill_cus[i] < 8 || prefill_cus[i] % 8 || n_cu - prefill_cus[i] < 8)
            return fail(MW_ERR_INVALID_ARG, "mw_engine_create: prefill CUs %d must be a multiple of 8 leaving >= 8 of %d",
                        prefill_cus[i], n_cu);
    int prev = 0;
    MW_HIP_TRY(hipGetDevice(&prev));
    MW_HIP_TRY(hipSetDevice(device));
    mw_engine *e = new (std::nothrow) mw_engine();
    if (!e) {
        (void)hipSetDevice(prev);
        return fail(MW_ERR_INVALID_ARG, "mw_engine_create: out of host memory");
    }
    e->device = device;
    e->n = n;
    size_t free0 = 0, free1 = 0, total = 0;
    (void)hipDeviceSynchronize();
    MW_HIP_TRY(hipMemGetInfo(&free0, &total));
    const clk::time_point t0 = clk::now();
    // the same bit layout as mw_partition_create: mask bit c selects a CU of
    // XCD c % 8, so the first 8k bits give k CUs on every XCD
    const int words = (n_cu + 31) / 32;
    mw_status st = MW_OK;
    for (int i = 0; i < n && st == MW_OK; ++i) {
        uint32_t pm[8] = {0}, dm[8] = {0};
        for (int c = 0; c < n_cu; ++c) (c < prefill_cus[i] ? pm : dm)[c / 32] |= 1u << (c % 32);
        e->prefill_cus[i] = prefill_cus[i];
        e->decode_cus[i] = n_cu - prefill_cus[i];
        st = masked_stream(words, pm, &e->prefill[i]);
        if (st == MW_OK) st = masked_stream(words, dm, &e->decode[i]);
    }
    if (st == MW_OK) {
        uint32_t all[8] = {0};
        for (int c = 0; c < n_cu; ++c) all[c / 32] |= 1u << (c % 32);
        st = masked_stream(words, all, &e->whole);
    }
    e->create_ms = ms_since(t0);
    if (st == MW_OK && hipMemGetInfo(&free1, &total) == hipSuccess)
        e->mem_bytes = static_cast<int64_t>(free0) - static_cast<int64_t>(free1);
    (void)hipSetDevice(prev);
    if (st != MW_OK) {
        destroy_streams(e);
        delete e;
        return st;
    }
    *out = e;
    return MW_OK;
}

mw_status mw_engine_destroy(mw_engine *eng) {
    if (!eng) return MW_OK;
    hipError_t err = hipSuccess;
    for (int i = 0; i < eng->n; ++i) {
        const hipError_t a = hipStreamSynchronize(eng->prefill[i]), b = hipStreamSynchronize(eng->decode[i]);
        if (err == hipSuccess) err = a != hipSuccess ? a : b;
    }
    const hipError_t c = hipStreamSynchronize(eng->whole);
    if (err == hipSuccess) err = c;
    destroy_graphs(eng);
    destroy_streams(eng);
    delete eng;
    if (err != hipSuccess) return fail(MW_ERR_HIP, "mw_engine_destroy: %s", hipGetErrorString(err));
    return MW_OK;
}

mw_status mw_engine_streams(const mw_engine *eng, int32_t config, mw_stream *prefill, mw_stream *decode) {
    if (!eng || config < -1 || config >= eng->n) return fail(MW_ERR_INVALID_ARG, "mw_engine_streams: bad arguments");
    if (prefill) *prefill = config < 0 ? eng->whole : eng->prefill[config];
    if (decode) *decode = config < 0 ? eng->whole : eng->decode[config];
    return MW_OK;
}

mw_status mw_engine_memory(const mw_engine *eng, int64_t *device_bytes, double *create_ms) {
    if (!eng) return fail(MW_ERR_INVALID_ARG, "mw_engine_memory: NULL engine");
    if (device_bytes) *device_bytes = eng->mem_bytes;
    if (create_ms) *create_ms = eng->create_ms;
    return MW_OK;
}

mw_status mw_engine_run(mw_engine *eng, const mw_decode_args *dec, const mw_prefill_args *pre,
                        const mw_engine_plan *plan, mw_engine_stats *stats) {
    mw_status st = check_args(eng, dec, pre, plan);
    if (st != MW_OK) return st;
    if (!stats) return fail(MW_ERR_INVALID_ARG, "mw_engine_run: NULL stats");
    const int cfg = plan->config;
    hipStream_t ds = eng->decode[cfg], ps = eng->prefill[cfg];
    int prev = 0;
    MW_HIP_TRY(hipGetDevice(&prev));
    MW_HIP_TRY(hipSetDevice(eng->device));
    MW_HIP_TRY(hipStreamSynchronize(ds));
    MW_HIP_TRY(hipStreamSynchronize(ps));
    MW_HIP_TRY(hipStreamSynchronize(eng->whole));

    // a decode iteration as one graph launch: looked up or captured (on the
    // partition's decode stream) before anything is timed
    hipGraphExec_t dgraph = nullptr;
    if (plan->decode_graph) {
        std::vector<unsigned char> key = graph_key(dec, plan->decode_layers);
        for (const mw_engine::Graph &g : eng->graphs)
            if (g.config == cfg && g.layers == plan->decode_layers && g.key == key) dgraph = g.exec;
        if (!dgraph) {
            mw_engine::Graph g{cfg, plan->decode_layers, key, nullptr, nullptr, 0, 0.0};
            size_t f0 = 0, f1 = 0, tot = 0;
            MW_HIP_TRY(hipDeviceSynchronize());
            MW_HIP_TRY(hipMemGetInfo(&f0, &tot));
            const clk::time_point t0 = clk::now();
            MW_HIP_TRY(hipStreamBeginCapture(ds, hipStreamCaptureModeThreadLocal));
            for (int l = 0; l < plan->decode_layers && st == MW_OK; ++l)
                st = mw_decode_attn(dec->pool, &dec->shape, dec->batch, dec->h_seq_lens, dec->d_seq_lens,
                                    dec->d_block_table, dec->bt_stride, dec->d_q, dec->d_out, dec->d_workspace,
                                    dec->workspace_bytes, dec->chunk_pages, ds, nullptr);
            const hipError_t ec = hipStreamEndCapture(ds, &g.graph);
            if (st == MW_OK && ec != hipSuccess)
                st = fail(MW_ERR_HIP, "hipStreamEndCapture failed: %s", hipGetErrorString(ec));
            if (st == MW_OK && hipGraphInstantiate(&g.exec, g.graph, nullptr, nullptr, 0) != hipSuccess)
                st = fail(MW_ERR_HIP, "hipGraphInstantiate failed");
            if (st == MW_OK && hipGraphUpload(g.exec, ds) != hipSuccess) st = fail(MW_ERR_HIP, "hipGraphUpload failed");
            if (st == MW_OK && hipStreamSynchronize(ds) != hipSuccess) st = fail(MW_ERR_HIP, "graph upload failed");
            if (st != MW_OK) {
                if (g.exec) (void)hipGraphExecDestroy(g.exec);
                if (g.graph) (void)hipGraphDestroy(g.graph);
                (void)hipGetLastError();
                (void)hipSetDevice(prev);
                return st;
            }
            g.capture_ms = ms_since(t0);
            if (hipMemGetInfo(&f1, &tot) == hipSuccess) g.bytes = static_cast<int64_t>(f0) - static_cast<int64_t>(f1);
            eng->graphs.push_back(g);
            dgraph = g.exec;
        }
    }
    const int calls_per_iter = dgraph ? 1 : plan->decode_layers;

    // all events up front: creating one inside the loop would add host time there
    EventPool pool;
    const size_t n_events = 1 + 2 * (static_cast<size_t>(plan->decode_iters) * calls_per_iter +
                                     static_cast<size_t>(plan->prefill_layers));
    for (size_t i = 0; i < n_events && st == MW_OK; ++i) {
        hipEvent_t e;
        if (hipEventCreate(&e) != hipSuccess) {
            st = fail(MW_ERR_HIP, "hipEventCreate failed");
            break;
        }
        pool.all.push_back(e);
    }
    if (st != MW_OK) {
        (void)hipSetDevice(prev);
        return st;
    }
    hipEvent_t ref;
    st = pool.get(&ref);
    std::vector<Span> dspan, pspan;     // per call
    std::vector<int> pstream;           // per prefill call: 0 = partition, 1 = whole device
    std::vector<hipEvent_t> iter_end;   // per decode iteration
    double host_ms = 0.0, dec_host_ms = 0.0;
    int prefill_batches = 0, switched = 0;
    double switch_host_us = -1.0;
    int switch_at = -1;                 // first prefill call on the whole device

    auto span_around = [&](hipStream_t s, std::vector<Span> &v, auto launch) -> mw_status {
        Span sp;
        mw_status r = pool.get(&sp.start);
        if (r == MW_OK) r = pool.get(&sp.end);
        if (r != MW_OK) return r;
        MW_HIP_TRY(hipEventRecord(sp.start, s));
        r = launch(s);
        if (r != MW_OK) return r;
        MW_HIP_TRY(hipEventRecord(sp.end, s));
        v.push_back(sp);
        return MW_OK;
    };
    auto decode_call = [&](hipStream_t s) {
        return mw_decode_attn(dec->pool, &dec->shape, dec->batch, dec->h_seq_lens, dec->d_seq_lens,
                              dec->d_block_table, dec->bt_stride, dec->d_q, dec->d_out, dec->d_workspace,
                              dec->workspace_bytes, dec->chunk_pages, s, nullptr);
    };
    auto prefill_call = [&](hipStream_t s) {
        if (pre->d_workspace)
            return mw_prefill_attn_ws(pre->pool, &pre->shape, pre->batch, pre->h_new_lens, pre->h_prefix_lens,
                                      pre->d_qo_indptr, pre->d_prefix_lens, pre->d_block_table, pre->bt_stride,
                                      pre->d_q, pre->d_out, pre->d_workspace, pre->workspace_bytes, s, nullptr);
        return mw_prefill_attn(pre->pool, &pre->shape, pre->batch, pre->h_new_lens, pre->h_prefix_lens,
                               pre->d_qo_indptr, pre->d_prefix_lens, pre->d_block_table, pre->bt_stride, pre->d_q,
                               pre->d_out, s, nullptr);
    };
    auto graph_call = [&](hipStream_t s) -> mw_status {
        MW_HIP_TRY(hipGraphLaunch(dgraph, s));
        return MW_OK;
    };
    auto launch_iteration = [&]() -> mw_status {
        const clk::time_point t0 = clk::now();
        for (int l = 0; l < calls_per_iter; ++l) {
            mw_status r = dgraph ? span_around(ds, dspan, graph_call) : span_around(ds, dspan, decode_call);
            if (r != MW_OK) return r;
        }
        iter_end.push_back(dspan.back().end);
        const double dt = ms_since(t0);
        host_ms += dt;
        dec_host_ms += dt;
        return MW_OK;
    };
    hipStream_t pcur = ps;
    auto launch_layers = [&](int k) -> mw_status {
        const clk::time_point t0 = clk::now();
        for (int l = 0; l < k; ++l) {
            mw_status r = span_around(pcur, pspan, prefill_call);
            if (r != MW_OK) return r;
            pstream.push_back(pcur == eng->whole ? 1 : 0);
        }
        ++prefill_batches;
        host_ms += ms_since(t0);
        return MW_OK;
    };

    // the reference point: both streams idle; everything is timed from here
    if (st == MW_OK && hipEventRecord(ref, ds) != hipSuccess) st = fail(MW_ERR_HIP, "hipEventRecord failed");
    if (st == MW_OK && hipStreamWaitEvent(ps, ref, 0) != hipSuccess) st = fail(MW_ERR_HIP, "hipStreamWaitEvent failed");

    if (st == MW_OK && plan->policy == MW_ENGINE_BLOCKING) {
        for (int it = 0; it < plan->decode_iters && st == MW_OK; ++it) {
            st = launch_iteration();
            if (st == MW_OK && it == 0) st = launch_layers(plan->prefill_layers);
            if (st == MW_OK && hipEventSynchronize(iter_end.back()) != hipSuccess)
                st = fail(MW_ERR_HIP, "hipEventSynchronize failed");
        }
    } else if (st == MW_OK) {
        const int npl = std::min(plan->layers_per_launch, plan->prefill_layers);
        int iters_done = 0, launched = 0, completed = 0;
        bool dec_running = false;
        st = launch_iteration();
        dec_running = st == MW_OK;
        if (st == MW_OK) {
            st = launch_layers(npl);
            launched = npl;
        }
        while (st == MW_OK && (iters_done < plan->decode_iters || completed < plan->prefill_layers)) {
            if (dec_running) {
                const hipError_t q = hipEventQuery(iter_end.back());
                if (q == hipSuccess) {
                    dec_running = false;
                    ++iters_done;
                    if (iters_done < plan->decode_iters) {
                        st = launch_iteration();
                        dec_running = true;
                    } else if (plan->switch_on_decode_end && launched < plan->prefill_layers && pcur == ps) {
                        // decode is over: later layers run on the whole device,
                        // after the layers already queued on the partition
                        const clk::time_point t0 = clk::now();
                        hipEvent_t last = pspan.back().end;
                        if (hipStreamWaitEvent(eng->whole, last, 0) != hipSuccess)
                            st = fail(MW_ERR_HIP, "hipStreamWaitEvent failed");
                        pcur = eng->whole;
                        switch_at = launched;
                        switch_host_us = ms_since(t0) * 1e3;
                        if (st == MW_OK) {
                            const int k = std::min(npl, plan->prefill_layers - launched);
                            st = launch_layers(k);
                            launched += k;
                        }
                    }
                } else if (q != hipErrorNotReady) {
                    st = fail(MW_ERR_HIP, "hipEventQuery failed: %s", hipGetErrorString(q));
                }
            }
            while (st == MW_OK && completed < launched) {
                const hipError_t q = hipEventQuery(pspan[completed].end);
                if (q == hipErrorNotReady) break;
                if (q != hipSuccess) st = fail(MW_ERR_HIP, "hipEventQuery failed: %s", hipGetErrorString(q));
                ++completed;
            }
            if (st == MW_OK && launched < plan->prefill_layers && launched - completed < npl) {
                const int k = std::min(npl, plan->prefill_layers - launched);
                st = launch_layers(k);
                launched += k;
            }
        }
    }
    // every launched call completes before the stats are read (also on error)
    (void)hipStreamSynchronize(ds);
    (void)hipStreamSynchronize(ps);
    (void)hipStreamSynchronize(eng->whole);
    if (st == MW_OK) {
        hipError_t le = hipGetLastError();
        if (le != hipSuccess) st = fail(MW_ERR_HIP, "mw_engine_run: %s", hipGetErrorString(le));
    }
    if (st != MW_OK) {
        (void)hipSetDevice(prev);
        return st;
    }

    auto at = [&](hipEvent_t e) {
        float ms = 0.f;
        (void)hipEventElapsedTime(&ms, ref, e);
        return static_cast<double>(ms);
    };
    mw_engine_stats s{};
    // decode stream
    double busy = 0.0, first = 1e30, last = 0.0, gap_max = 0.0, iter_sum = 0.0;
    const size_t L = static_cast<size_t>(calls_per_iter);
    for (size_t i = 0; i < dspan.size(); ++i) {
        const double a = at(dspan[i].start), b = at(dspan[i].end);
        busy += b - a;
        first = std::min(first, a);
        last = std::max(last, b);
    }
    for (size_t it = 0; it * L < dspan.size(); ++it) {
        const double a = at(dspan[it * L].start), b = at(dspan[it * L + L - 1].end);
        iter_sum += b - a;
        if (it > 0) gap_max = std::max(gap_max, a - at(dspan[it * L - 1].end));
    }
    s.decode_busy_ms = busy;
    s.decode_bubble = last > first ? 1.0 - busy / (last - first) : 0.0;
    s.decode_gap_ms_max = gap_max;
    s.decode_iter_ms_mean = iter_sum / static_cast<double>(dspan.size() / L);
    double wall = last;
    // prefill timeline (partition then, after a switch, the whole device)
    busy = 0.0;
    first = 1e30;
    last = 0.0;
    for (size_t i = 0; i < pspan.size(); ++i) {
        const double a = at(pspan[i].start), b = at(pspan[i].end);
        busy += b - a;
        first = std::min(first, a);
        last = std::max(last, b);
        switched += pstream[i];
    }
    s.prefill_busy_ms = busy;
    s.prefill_bubble = last > first ? 1.0 - busy / (last - first) : 0.0;
    s.prefill_end_ms = last;
    wall = std::max(wall, last);
    s.wall_ms = wall;
    s.bubble_ratio = 0.5 * (s.decode_bubble + s.prefill_bubble);
    s.switch_gap_ms = switch_at > 0 ? at(pspan[switch_at].start) - at(pspan[switch_at - 1].end) : -1.0;
    s.switch_host_us = switch_host_us;
    s.host_launch_ms = host_ms;
    s.decode_launch_us_mean = 1e3 * dec_host_ms / static_cast<double>(iter_end.size());
    s.prefill_batches = prefill_batches;
    s.switched_layers = switched;
    *stats = s;
    for (int ph = 0; ph < 2; ++ph) {
        const std::vector<Span> &v = ph == 0 ? dspan : pspan;
        std::vector<double> &t = eng->timeline[ph];
        t.clear();
        for (size_t i = 0; i < v.size(); ++i) {
            t.push_back(at(v[i].start));
            t.push_back(at(v[i].end));
            t.push_back(ph == 1 ? static_cast<double>(pstream[i]) : 0.0);
        }
    }
    (void)hipSetDevice(prev);
    return MW_OK;
}

mw_status mw_engine_graphs(const mw_engine *eng, int32_t *n_graphs, int64_t *device_bytes, double *capture_ms) {
    if (!eng) return fail(MW_ERR_INVALID_ARG, "mw_engine_graphs: NULL engine");
    int64_t b = 0;
    double ms = 0.0;
    for (const mw_engine::Graph &g : eng->graphs) {
        b += g.bytes;
        ms += g.capture_ms;
    }
    if (n_graphs) *n_graphs = static_cast<int32_t>(eng->graphs.size());
    if (device_bytes) *device_bytes = b;
    if (capture_ms) *capture_ms = ms;
    return MW_OK;
}

mw_status mw_engine_timeline(const mw_engine *eng, int32_t phase, double *out, int32_t capacity,
                             int32_t *n_calls) {
    if (!eng || (phase != 0 && phase != 1) || capacity < 0 || (capacity > 0 && !out) || !n_calls)
        return fail(MW_ERR_INVALID_ARG, "mw_engine_timeline: bad arguments");
    const std::vector<double> &t = eng->timeline[phase];
    const int32_t n = static_cast<int32_t>(t.size() / 3);
    *n_calls = n;
    std::copy(t.begin(), t.begin() + 3 * static_cast<size_t>(std::min(n, capacity)), out);
    return MW_OK;
}

}  // extern "C"
