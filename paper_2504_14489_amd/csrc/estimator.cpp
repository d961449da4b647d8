// Contention-tolerant estimator (paper Sec. 3.3): solo-run latency models of
// Eqs. (1)-(2) fitted by least squares, the contention guard's grid of maximum
// decode slowdowns, and the dispatcher's prefill-layer count (Sec. 3.4).
// Host code only.
#include <algorithm>
#include <cmath>
#include <map>
#include <queue>
#include <set>
#include <tuple>
#include <vector>

#include "mw_internal.h"

using namespace mw;

namespace {

constexpr int kPrefillTerms = 4;  // sum n^2, sum n r, sum n, 1
constexpr int kDecodeTerms = 3;   // sum r, bs, 1

struct Model {
    int terms = 0;
    std::vector<double> x;  // samples x terms, row-major
    std::vector<double> t;  // measured ms
    double theta[4] = {0, 0, 0, 0};
    bool fitted = false;
};

// Least squares of the relative error: minimise sum_j ((x_j . th - t_j) / t_j)^2,
// i.e. ordinary least squares on rows x_j / t_j against 1.  Columns are scaled to
// unit maximum, then Householder QR; a column that is zero in every sample (a
// term the samples never exercise) gets coefficient 0.  Returns false when the
// remaining columns are linearly dependent.
bool fit_relative(Model &m) {
    const int n = static_cast<int>(m.t.size()), k = m.terms;
    std::vector<double> a(static_cast<size_t>(n) * k), b(n, 1.0), scale(k, 0.0);
    for (int j = 0; j < n; ++j)
        for (int c = 0; c < k; ++c) {
            a[j * k + c] = m.x[j * k + c] / m.t[j];
            scale[c] = std::max(scale[c], std::fabs(a[j * k + c]));
        }
    std::vector<int> cols;
    for (int c = 0; c < k; ++c)
        if (scale[c] > 0) cols.push_back(c);
    const int kk = static_cast<int>(cols.size());
    if (kk == 0 || n < kk) return false;
    // working matrix of the used, scaled columns (column-major for the reflections)
    std::vector<double> w(static_cast<size_t>(n) * kk);
    for (int c = 0; c < kk; ++c)
        for (int j = 0; j < n; ++j) w[c * n + j] = a[j * k + cols[c]] / scale[cols[c]];
    std::vector<double> rdiag(kk);
    for (int c = 0; c < kk; ++c) {
        double norm = 0;
        for (int j = c; j < n; ++j) norm += w[c * n + j] * w[c * n + j];
        norm = std::sqrt(norm);
        if (norm == 0) return false;
        const double alpha = w[c * n + c] > 0 ? -norm : norm;
        // reflector v = x - alpha e_c, applied as I - 2 v v^T / (v^T v)
        w[c * n + c] -= alpha;
        double vv = 0;
        for (int j = c; j < n; ++j) vv += w[c * n + j] * w[c * n + j];
        for (int d = c + 1; d < kk; ++d) {
            double dot = 0;
            for (int j = c; j < n; ++j) dot += w[c * n + j] * w[d * n + j];
            const double f = 2 * dot / vv;
            for (int j = c; j < n; ++j) w[d * n + j] -= f * w[c * n + j];
        }
        double dot = 0;
        for (int j = c; j < n; ++j) dot += w[c * n + j] * b[j];
        const double f = 2 * dot / vv;
        for (int j = c; j < n; ++j) b[j] -= f * w[c * n + j];
        rdiag[c] = alpha;
    }
    double rmax = 0;
    for (double r : rdiag) rmax = std::max(rmax, std::fabs(r));
    for (double r : rdiag)
        if (std::fabs(r) <= 1e-12 * rmax) return false;
    // back substitution R th' = (Q^T b)[0:kk]; R's strict upper part sits in w
    std::vector<double> th(kk);
    for (int c = kk - 1; c >= 0; --c) {
        double s = b[c];
        for (int d = c + 1; d < kk; ++d) s -= w[d * n + c] * th[d];
        th[c] = s / rdiag[c];
    }
    for (int c = 0; c < k; ++c) m.theta[c] = 0;
    for (int c = 0; c < kk; ++c) m.theta[cols[c]] = th[c] / scale[cols[c]];
    m.fitted = true;
    return true;
}

bool prefill_terms(int32_t batch, const int32_t *nl, const int32_t *rl, double out[4]) {
    double s2 = 0, snr = 0, sn = 0;
    for (int32_t i = 0; i < batch; ++i) {
        if (nl[i] < 1 || rl[i] < 0) return false;
        const double n = nl[i], r = rl[i];
        s2 += n * n;
        snr += n * r;
        sn += n;
    }
    out[0] = s2;
    out[1] = snr;
    out[2] = sn;
    out[3] = 1;
    return true;
}

bool decode_terms(int32_t batch, const int32_t *lens, double out[4]) {
    double sr = 0;
    for (int32_t i = 0; i < batch; ++i) {
        if (lens[i] < 1) return false;
        sr += lens[i] - 1;
    }
    out[0] = sr;
    out[1] = batch;
    out[2] = 1;
    out[3] = 0;
    return true;
}

// The library's prefill launch on `cus` CUs, from the lengths: its kernel path
// (0: 8-wave blocks of 64 positions, one work-group per CU; 1: 4-wave blocks
// of 32 positions, two work-groups per CU, with the key-range split when its
// plan cuts, as a call with a workspace makes it) and its load-imbalance
// factor: the latest CU's finishing time over the time of the same work spread
// evenly over the CUs.  The work-groups are taken in dispatch order (grid x
// fastest, then the sequence) and each goes to the CU slot that frees first,
// all CUs' first slots before any second one; a work-group's work is its key
// tiles (64 keys each), summed over the blocks it takes.  A CU that holds a
// single work-group of a two-per-CU launch runs it at 0.9 of a shared CU's
// rate: two work-groups sharing a CU each run about 1.8 times slower than one
// alone (measured), i.e. the pair moves 2 / 1.8 times the work.
struct PrefillLaunch {
    int path;
    double kappa;
};

PrefillLaunch prefill_launch(int32_t batch, const int32_t *nl, const int32_t *rl, int hkv, int group, int64_t cus) {
    PrefillPlan pl;
    prefill_plan_lengths(batch, nl, hkv, group, cus, true, &pl);
    if (pl.waves == 4) prefill_split_plan(batch, nl, rl, hkv * group, cus, &pl);
    const int bm = pl.waves == 4 ? 32 : 64;
    const int per_cu = pl.waves == 4 ? 2 : 1;
    const int64_t heads = static_cast<int64_t>(pl.hkv) * pl.n_hgroups;
    int64_t max_n = 0;
    for (int32_t b = 0; b < batch; ++b) max_n = std::max<int64_t>(max_n, nl[b]);
    std::vector<double> work;
    for (int32_t b = 0; b < batch; ++b) {
        const int n = nl[b], r = rl[b];
        const int nqb = (n + bm - 1) / bm;
        auto tiles = [&](int q) { return (r + std::min(q * bm + bm, n) + 63) / 64; };
        if (pl.pieces > 1) {  // split kernel: x = unit * pieces + piece, single blocks
            const int64_t gx = (max_n + bm - 1) / bm * heads * pl.pieces;
            for (int64_t x = 0; x < gx; ++x) {
                const int64_t pair = x / pl.pieces / heads;
                const int piece = static_cast<int>(x % pl.pieces);
                if (pair >= nqb) continue;
                const int ntb = tiles(nqb - 1 - static_cast<int>(pair));
                const int np = prefill_pieces(ntb, pl.piece_tiles, pl.pieces);
                if (piece >= np) continue;
                work.push_back((piece + 1) * ntb / np - piece * ntb / np);
            }
        } else {
            for (int64_t x = 0; x < pl.gx; ++x) {
                const int pair = static_cast<int>(x / heads);
                const int last = nqb - 1 - pair;
                if (pl.paired ? pair >= (nqb + 1) / 2 : pair >= nqb) continue;
                work.push_back(tiles(last) + (pl.paired && pair != last ? tiles(pair) : 0));
            }
        }
    }
    double total = 0;
    for (double w : work) total += w;
    if (!(total > 0)) return {pl.waves == 4 ? 1 : 0, 1.0};
    // Dispatch: each work-group goes to a slot that frees within a window (5%
    // of the mean work-group's work) of the earliest free time, and among those
    // to the CU holding the fewest work-groups so far, then the lower slot
    // index, then the lower CU: work-groups a tile or two apart finish together
    // on the GPU and the next ones spread over the CUs that freed.  The
    // earliest free time never decreases, so a slot inside the window stays
    // there until it takes a work-group.
    const double window = 0.05 * total / static_cast<double>(work.size());
    const int64_t nslots = per_cu * cus;  // slot = k * cus + c
    std::vector<double> t_free(nslots, 0.0);
    std::vector<char> in_window(nslots, 0);
    using Timed = std::pair<double, int64_t>;  // free time, slot
    std::priority_queue<Timed, std::vector<Timed>, std::greater<Timed>> later;
    std::set<std::tuple<int, int, int64_t>> ready;  // (work-groups on the CU, slot index, CU)
    std::multiset<double> ready_t;
    for (int64_t sl = 0; sl < nslots; ++sl) later.emplace(0.0, sl);
    std::vector<double> load(cus, 0.0);
    std::vector<int> count(cus, 0);
    for (double w : work) {
        double t0 = later.empty() ? INFINITY : later.top().first;
        if (!ready_t.empty()) t0 = std::min(t0, *ready_t.begin());
        while (!later.empty() && later.top().first <= t0 + window) {
            const int64_t sl = later.top().second;
            later.pop();
            ready.emplace(count[sl % cus], static_cast<int>(sl / cus), sl % cus);
            ready_t.insert(t_free[sl]);
            in_window[sl] = 1;
        }
        const auto pick = *ready.begin();
        ready.erase(ready.begin());
        const int k = std::get<1>(pick);
        const int64_t c = std::get<2>(pick), sl = k * cus + c;
        ready_t.erase(ready_t.find(t_free[sl]));
        in_window[sl] = 0;
        for (int k2 = 0; k2 < per_cu; ++k2)  // the CU's other slots in the window move to its new count
            if (k2 != k && in_window[k2 * cus + c]) {
                ready.erase(std::make_tuple(count[c], k2, c));
                ready.emplace(count[c] + 1, k2, c);
            }
        ++count[c];
        load[c] += w;
        t_free[sl] += w;
        later.emplace(t_free[sl], sl);
    }
    double t_max = 0;
    for (int64_t c = 0; c < cus; ++c)
        t_max = std::max(t_max, load[c] / (per_cu == 2 && count[c] == 1 ? 0.9 : 1.0));
    return {pl.waves == 4 ? 1 : 0, t_max * static_cast<double>(cus) / total};
}

int cell(int64_t x, int64_t base) {
    int k = 0;
    for (int64_t v = 1; v < x; v *= base) ++k;
    return k;
}

}  // namespace

struct mw_predictor {
    // (phase, cus) -> model; phase 0 = prefill (8-wave path, or every prefill
    // call without a launch shape), 1 = decode, 2 = prefill on the 4-wave path
    std::map<std::pair<int, int>, Model> models;
    int hkv = 0, group = 0;  // launch shape (0: plain Eq. (1) terms)
};

struct mw_guard {
    std::map<std::tuple<int, int, int, int, int>, double> cells;  // cus, cells of the four counts
};

extern "C" {

mw_status mw_predictor_create(mw_predictor **out) {
    if (!out) return fail(MW_ERR_INVALID_ARG, "mw_predictor_create: NULL out");
    *out = new mw_predictor();
    return MW_OK;
}

mw_status mw_predictor_destroy(mw_predictor *p) {
    delete p;
    return MW_OK;
}

static mw_status add_sample(mw_predictor *p, int phase, int32_t cus, const double *x, int terms, double ms,
                            const char *who) {
    if (!(ms > 0) || !std::isfinite(ms)) return fail(MW_ERR_INVALID_ARG, "%s: ms must be positive and finite", who);
    Model &m = p->models[{phase, cus}];
    m.terms = terms;
    m.x.insert(m.x.end(), x, x + terms);
    m.t.push_back(ms);
    m.fitted = false;
    return MW_OK;
}

mw_status mw_predictor_set_launch_shape(mw_predictor *p, int32_t num_q_heads, int32_t num_kv_heads) {
    const char *who = "mw_predictor_set_launch_shape";
    if (!p || num_kv_heads < 1 || num_q_heads < 1 || num_q_heads % num_kv_heads)
        return fail(MW_ERR_INVALID_ARG, "%s: bad arguments", who);
    for (const auto &kv : p->models)
        if (kv.first.first != 1 && !kv.second.t.empty())
            return fail(MW_ERR_INVALID_ARG, "%s: prefill samples were added before the shape", who);
    p->hkv = num_kv_heads;
    p->group = num_q_heads / num_kv_heads;
    return MW_OK;
}

// Eq. (1) terms of a prefill call and the model they belong to: with a launch
// shape, the n^2, n r and n terms are scaled by the launch's load-imbalance
// factor and the kernel path picks the model.
static bool prefill_sample(const mw_predictor *p, int32_t cus, int32_t batch, const int32_t *nl, const int32_t *rl,
                           double x[4], int *phase) {
    if (!prefill_terms(batch, nl, rl, x)) return false;
    *phase = 0;
    if (p->hkv > 0) {
        const PrefillLaunch l = prefill_launch(batch, nl, rl, p->hkv, p->group, cus);
        for (int c = 0; c < 3; ++c) x[c] *= l.kappa;
        *phase = l.path == 0 ? 0 : 2;
    }
    return true;
}

mw_status mw_predictor_add_prefill(mw_predictor *p, int32_t cus, int32_t batch, const int32_t *new_lens,
                                   const int32_t *prefix_lens, double ms) {
    const char *who = "mw_predictor_add_prefill";
    double x[4];
    int phase = 0;
    if (!p || cus < 1 || batch < 1 || !new_lens || !prefix_lens ||
        !prefill_sample(p, cus, batch, new_lens, prefix_lens, x, &phase))
        return fail(MW_ERR_INVALID_ARG, "%s: bad arguments", who);
    return add_sample(p, phase, cus, x, kPrefillTerms, ms, who);
}

mw_status mw_predictor_add_decode(mw_predictor *p, int32_t cus, int32_t batch, const int32_t *seq_lens, double ms) {
    const char *who = "mw_predictor_add_decode";
    double x[4];
    if (!p || cus < 1 || batch < 1 || !seq_lens || !decode_terms(batch, seq_lens, x))
        return fail(MW_ERR_INVALID_ARG, "%s: bad arguments", who);
    return add_sample(p, 1, cus, x, kDecodeTerms, ms, who);
}

mw_status mw_predictor_fit(mw_predictor *p) {
    if (!p) return fail(MW_ERR_INVALID_ARG, "mw_predictor_fit: NULL predictor");
    int fitted = 0;
    for (auto &kv : p->models) {
        Model &m = kv.second;
        if (static_cast<int>(m.t.size()) < m.terms) continue;
        if (!fit_relative(m)) {
            // the 4-wave path's few samples on a small partition (calls that
            // short are all alike) may leave its model open: that path then
            // uses the 8-wave path's model
            if (kv.first.first == 2) continue;
            return fail(MW_ERR_INVALID_ARG, "mw_predictor_fit: the %s samples on %d CUs do not determine the model",
                        kv.first.first == 1 ? "decode" : kv.first.first == 0 ? "prefill" : "4-wave prefill",
                        kv.first.second);
        }
        ++fitted;
    }
    return fitted ? MW_OK : fail(MW_ERR_NOT_READY, "mw_predictor_fit: no model has enough samples");
}

static mw_status predict(const mw_predictor *p, int phase, int32_t cus, const double *x, double *ms,
                         const char *who) {
    auto it = p->models.find({phase, cus});
    if ((it == p->models.end() || !it->second.fitted) && phase != 1)  // the other prefill path's model
        it = p->models.find({phase == 0 ? 2 : 0, cus});
    if (it == p->models.end() || !it->second.fitted)
        return fail(MW_ERR_NOT_READY, "%s: no fitted model for %d CUs", who, cus);
    double s = 0;
    for (int c = 0; c < it->second.terms; ++c) s += it->second.theta[c] * x[c];
    *ms = s;
    return MW_OK;
}

mw_status mw_predictor_prefill_ms(const mw_predictor *p, int32_t cus, int32_t batch, const int32_t *new_lens,
                                  const int32_t *prefix_lens, double *ms) {
    const char *who = "mw_predictor_prefill_ms";
    double x[4];
    int phase = 0;
    if (!p || !ms || cus < 1 || batch < 1 || !new_lens || !prefix_lens ||
        !prefill_sample(p, cus, batch, new_lens, prefix_lens, x, &phase))
        return fail(MW_ERR_INVALID_ARG, "%s: bad arguments", who);
    return predict(p, phase, cus, x, ms, who);
}

mw_status mw_predictor_decode_ms(const mw_predictor *p, int32_t cus, int32_t batch, const int32_t *seq_lens,
                                 double *ms) {
    const char *who = "mw_predictor_decode_ms";
    double x[4];
    if (!p || !ms || batch < 1 || !seq_lens || !decode_terms(batch, seq_lens, x))
        return fail(MW_ERR_INVALID_ARG, "%s: bad arguments", who);
    return predict(p, 1, cus, x, ms, who);
}

mw_status mw_predictor_coefficients(const mw_predictor *p, int32_t phase, int32_t cus, double theta[4]) {
    if (!p || !theta || phase < 0 || phase > 2)
        return fail(MW_ERR_INVALID_ARG, "mw_predictor_coefficients: bad arguments");
    auto it = p->models.find({phase, cus});
    if (it == p->models.end() || !it->second.fitted)
        return fail(MW_ERR_NOT_READY, "mw_predictor_coefficients: no fitted model for %d CUs", cus);
    for (int c = 0; c < 4; ++c) theta[c] = it->second.theta[c];
    return MW_OK;
}

mw_status mw_guard_create(mw_guard **out) {
    if (!out) return fail(MW_ERR_INVALID_ARG, "mw_guard_create: NULL out");
    *out = new mw_guard();
    return MW_OK;
}

mw_status mw_guard_destroy(mw_guard *g) {
    delete g;
    return MW_OK;
}

static bool guard_key(const mw_guard_key *k, std::tuple<int, int, int, int, int> *out) {
    if (!k || k->prefill_new < 0 || k->prefill_reused < 0 || k->decode_batch < 1 || k->decode_reused < 0 ||
        k->prefill_cus < 1)
        return false;
    *out = std::make_tuple(k->prefill_cus, cell(k->prefill_new, 4), cell(k->prefill_reused, 4),
                           cell(k->decode_batch, 2), cell(k->decode_reused, 4));
    return true;
}

mw_status mw_guard_add(mw_guard *g, const mw_guard_key *key, double slowdown) {
    std::tuple<int, int, int, int, int> c;
    if (!g || !guard_key(key, &c) || !(slowdown > 0) || !std::isfinite(slowdown))
        return fail(MW_ERR_INVALID_ARG, "mw_guard_add: bad arguments");
    auto it = g->cells.find(c);
    if (it == g->cells.end())
        g->cells.emplace(c, slowdown);
    else
        it->second = std::max(it->second, slowdown);
    return MW_OK;
}

mw_status mw_guard_lookup(const mw_guard *g, const mw_guard_key *key, double *slowdown) {
    std::tuple<int, int, int, int, int> c;
    if (!g || !slowdown || !guard_key(key, &c)) return fail(MW_ERR_INVALID_ARG, "mw_guard_lookup: bad arguments");
    auto it = g->cells.find(c);
    if (it != g->cells.end()) {
        *slowdown = it->second;
        return MW_OK;
    }
    double same = 0, all = 0;
    for (const auto &kv : g->cells) {
        all = std::max(all, kv.second);
        if (std::get<0>(kv.first) == std::get<0>(c)) same = std::max(same, kv.second);
    }
    *slowdown = same > 0 ? same : (all > 0 ? all : 1.0);
    return MW_OK;
}

mw_status mw_prefill_layers(double t_decode_ms, double t_prefill_ms, int32_t n_layers, int32_t *n_pl) {
    if (!n_pl || n_layers < 1 || !(t_decode_ms > 0) || !(t_prefill_ms > 0) || !std::isfinite(t_decode_ms) ||
        !std::isfinite(t_prefill_ms))
        return fail(MW_ERR_INVALID_ARG, "mw_prefill_layers: bad arguments");
    const double v = std::ceil(t_decode_ms * n_layers / t_prefill_ms);
    *n_pl = static_cast<int32_t>(std::min<double>(std::max(v, 1.0), n_layers));
    return MW_OK;
}

}  // extern "C"
