// The library's host logic on randomised inputs, for a build with
// AddressSanitizer and UndefinedBehaviorSanitizer: the decode and prefill
// launch planners, the page allocator and the estimator (with the prefill
// launch simulation).  Nothing here
// launches a kernel or touches a GPU: the device pointers are host addresses
// the planners only check for alignment.  Prints "ok" when every check holds.
#include <cstdio>
#include <cstdlib>
#include <vector>

#include "mw_internal.h"

namespace {

uint64_t g_state = 0x9E3779B97F4A7C15ull;
uint32_t next_u32() {  // xorshift64*
    g_state ^= g_state >> 12;
    g_state ^= g_state << 25;
    g_state ^= g_state >> 27;
    return static_cast<uint32_t>((g_state * 0x2545F4914F6CDD1Dull) >> 32);
}
int uniform(int lo, int hi) { return lo + static_cast<int>(next_u32() % static_cast<uint32_t>(hi - lo + 1)); }

int g_fail = 0;
void check(bool ok, const char *what, int it) {
    if (!ok) {
        std::fprintf(stderr, "check failed at iteration %d: %s (%s)\n", it, what, mw_last_error());
        ++g_fail;
    }
}

alignas(256) unsigned char g_fake[4096];  // stands in for device buffers: never dereferenced

void planners() {
    const int hkvs[4] = {1, 2, 4, 8};
    const int chunks[10] = {0, -1, 8, 16, 32, 64, 128, 256, 5, 300};
    for (int it = 0; it < 3000; ++it) {
        const int hkv = hkvs[uniform(0, 3)];
        const int group = uniform(1, 17);
        mw_kv_pool_desc desc{uniform(1, 1 << 14), 16, hkv, 128};
        mw_kv_pool *pool = nullptr;
        check(mw_kv_pool_create(&desc, g_fake, g_fake, &pool) == MW_OK, "pool create", it);
        const mw_attn_shape shape{hkv * group, hkv, 128, 0.0883883f};
        // decode: lengths on page edges, long and short, occasionally invalid;
        // a quarter of the batches are a few long sequences (equal or not),
        // whose segments the balanced split may pad to whole ranges
        const bool few_long = uniform(0, 3) == 0;
        const int batch = few_long ? uniform(1, 6) : uniform(0, 300);
        const bool equal = few_long && uniform(0, 1) == 0;
        std::vector<int32_t> lens(batch);
        int max_len = 1;
        for (int b = 0; b < batch; ++b) {
            const int kind = uniform(0, 9);
            if (few_long)
                lens[b] = equal && b > 0 ? lens[0] : uniform(2000, 70000);
            else
                lens[b] = kind == 0 ? 16 * uniform(1, 64) : kind == 1 ? uniform(1, 17) : uniform(1, 70000);
            max_len = lens[b] > max_len ? lens[b] : max_len;
        }
        if (batch > 0 && uniform(0, 49) == 0) lens[uniform(0, batch - 1)] = uniform(-3, 0);
        const int chunk = chunks[uniform(0, 9)];
        size_t bytes = 0;
        const mw_status st = mw_decode_workspace_size(&shape, batch, lens.data(), chunk, &bytes);
        const int stride = (max_len + 15) / 16 + uniform(-1, 3);
        mw_decode_args a{pool, shape, batch, lens.data(), reinterpret_cast<int32_t *>(g_fake),
                         reinterpret_cast<int32_t *>(g_fake), stride, g_fake, g_fake, g_fake, bytes, chunk};
        const int cus = uniform(0, 1) ? 8 * uniform(1, 32) : 0;
        mw::DecodePlan dp;
        const mw_status st2 = mw::decode_prepare(&a, cus, &dp, "decode_prepare");
        if (st == MW_OK && st2 == MW_OK) {
            check(dp.bytes <= bytes, "the workspace size covers the split of every CU count", it);
            check(dp.units >= 0 && dp.slots >= dp.units, "plan counts", it);
            check(dp.off_ml <= dp.off_meta && dp.off_meta <= dp.bytes, "workspace layout", it);
            // per-sequence chunk bases, or the balanced split's per-slot done flags
            const size_t meta = dp.per_unit > 0 ? static_cast<size_t>(dp.slots) * 4 : static_cast<size_t>(batch) * 4;
            check(dp.off_meta + meta <= dp.bytes, "workspace holds the flags", it);
            if (dp.aligned) {  // segments padded to whole ranges: one piece of one segment per unit
                int64_t padded = 0;
                for (int b = 0; b < batch; ++b)
                    padded += (static_cast<int64_t>(lens[b] + 15) / 16 + dp.per_unit - 1) / dp.per_unit * dp.per_unit;
                check(dp.per_unit >= 16 && dp.total == padded * hkv && dp.units * dp.per_unit == dp.total,
                      "aligned split covers every padded segment in whole ranges", it);
                check(cus > 0 && dp.units <= std::min<int64_t>(2 * cus, 512), "aligned split within the units", it);
            }
        }
        if (st != MW_OK) check(st2 != MW_OK, "a refused size is refused by the plan too", it);
        // prefill: varlen batches, prefixes, tables that are too short
        const int pb = uniform(0, 8);
        std::vector<int32_t> nl(pb), pl(pb);
        int max_tok = 1;
        for (int b = 0; b < pb; ++b) {
            nl[b] = uniform(0, 9) == 0 ? 0 : uniform(1, 5000);
            pl[b] = uniform(0, 3) == 0 ? 0 : uniform(0, 80000);
            max_tok = nl[b] + pl[b] > max_tok ? nl[b] + pl[b] : max_tok;
        }
        const int pstride = (max_tok + 15) / 16 + uniform(-1, 2);
        mw_prefill_args p{pool, shape, pb, nl.data(), pl.data(), reinterpret_cast<int32_t *>(g_fake),
                          reinterpret_cast<int32_t *>(g_fake), reinterpret_cast<int32_t *>(g_fake), pstride,
                          g_fake, g_fake};
        mw::PrefillPlan pp;
        const int pcus = 8 * uniform(1, 32);
        if (mw::prefill_prepare(&p, pcus, uniform(0, 1), &pp, "prefill_prepare") == MW_OK) {
            check(pp.gx >= 0 && (pp.waves == 4 || pp.waves == 8) && pp.group == group, "prefill plan", it);
            // the key-range split: at most the pieces the size call with no CU
            // count allows, pieces of at least 4 tiles, never cut 8-wave launches
            mw::prefill_split_plan(pb, nl.data(), pl.data(), shape.num_q_heads, pcus, &pp);
            size_t most = 0;
            check(mw_prefill_workspace_size(&shape, pb, nl.data(), pl.data(), 0, &most) == MW_OK, "size call", it);
            check(pp.split_bytes <= most, "the size with no CU count covers the plan", it);
            check(pp.pieces >= 1 && pp.pieces <= mw::kPrefillMaxPieces, "pieces", it);
            check(pp.pieces == 1 || (pp.waves == 4 && pp.piece_tiles >= mw::kPrefillMinPieceTiles), "cuts", it);
            for (int b = 0; b < pb; ++b)
                for (int qb = 0; 32 * qb < nl[b] && pp.pieces > 1; ++qb) {
                    const int nt = mw::prefill_block_tiles(pl[b], nl[b], qb);
                    const int k = mw::prefill_pieces(nt, pp.piece_tiles, pp.pieces);
                    // the last cut leaves the block's last two tiles (its diagonal) in the last piece
                    check(k == 1 || (k - 1) * nt / k <= nt - 2, "cut before the diagonal", it);
                    check(k == 1 || (k - 1) * nt / k <= (pl[b] + 32 * qb) / 64, "first tile of each piece visible", it);
                }
        }
        mw_kv_pool_destroy(pool);
    }
}

void allocator() {
    mw_kv_pool_desc desc{1000, 16, 2, 128};
    mw_kv_pool *pool = nullptr;
    check(mw_kv_pool_create(&desc, g_fake, g_fake, &pool) == MW_OK, "pool create", -1);
    std::vector<int32_t> held;
    for (int it = 0; it < 20000; ++it) {
        const int op = uniform(0, 9);
        int32_t n_free = 0;
        mw_kv_pool_num_free(pool, &n_free);
        check(n_free + static_cast<int>(held.size()) == 1000, "pages are conserved", it);
        if (op < 5) {
            const int n = uniform(0, 40);
            std::vector<int32_t> got(n);
            const mw_status st = mw_kv_pool_alloc(pool, n, got.data());
            if (st == MW_OK) held.insert(held.end(), got.begin(), got.end());
            else check(st == MW_ERR_OUT_OF_PAGES && n > n_free, "alloc refuses only when short", it);
        } else if (op < 9 && !held.empty()) {
            const int n = uniform(1, static_cast<int>(held.size()));
            std::vector<int32_t> back(held.end() - n, held.end());
            check(mw_kv_pool_free(pool, back.data(), n) == MW_OK, "free", it);
            held.resize(held.size() - n);
            if (uniform(0, 3) == 0) check(mw_kv_pool_free(pool, back.data(), 1) != MW_OK, "double free refused", it);
        } else {
            // renumber the free list: a permutation of the pages not held
            std::vector<uint8_t> is_held(1000, 0);
            for (int32_t x : held) is_held[x] = 1;
            std::vector<int32_t> order;
            for (int32_t x = 0; x < 1000; ++x)
                if (!is_held[x]) order.push_back(x);
            for (size_t i = order.size(); i > 1; --i) std::swap(order[i - 1], order[next_u32() % i]);
            check(mw_kv_pool_set_free_order(pool, order.data(), static_cast<int32_t>(order.size())) == MW_OK,
                  "set free order", it);
        }
    }
    mw_kv_pool_destroy(pool);
}

void estimator() {
    mw_predictor *p = nullptr;
    mw_guard *g = nullptr;
    check(mw_predictor_create(&p) == MW_OK && mw_guard_create(&g) == MW_OK, "estimator create", -1);
    for (int it = 0; it < 400; ++it) {
        const int cus = 8 * uniform(1, 32), batch = uniform(1, 12);
        std::vector<int32_t> n(batch), r(batch), L(batch);
        for (int b = 0; b < batch; ++b) {
            n[b] = uniform(1, 20000);
            r[b] = uniform(0, 100000);
            L[b] = uniform(1, 100000);
        }
        const double ms = 0.01 + uniform(0, 100000) * 1e-3;
        mw_predictor_add_prefill(p, cus, batch, n.data(), r.data(), ms);
        mw_predictor_add_decode(p, cus, batch, L.data(), ms);
        const mw_guard_key key{uniform(0, 1 << 20), uniform(0, 1 << 20), uniform(1, 512), uniform(0, 1 << 24), cus};
        mw_guard_add(g, &key, 1.0 + uniform(0, 1000) * 1e-3);
        double s = 0.0;
        check(mw_guard_lookup(g, &key, &s) == MW_OK && s >= 1.0, "guard lookup", it);
        if (it % 50 == 49) {
            mw_predictor_fit(p);
            double out = 0.0, th[4];
            mw_predictor_prefill_ms(p, cus, batch, n.data(), r.data(), &out);
            mw_predictor_decode_ms(p, cus, batch, L.data(), &out);
            mw_predictor_coefficients(p, uniform(0, 1), cus, th);
        }
        int32_t npl = 0;
        check(mw_prefill_layers(0.01 + ms, 0.02 + 2 * ms, uniform(1, 128), &npl) == MW_OK && npl >= 1,
              "prefill layers", it);
    }
    mw_predictor_destroy(p);
    mw_guard_destroy(g);
    // prefill models over the simulated launch: random shapes, batches and
    // partitions; every prediction of a fitted model is finite
    const int hkvs[4] = {1, 2, 4, 8};
    for (int shape = 0; shape < 6; ++shape) {
        mw_predictor *q = nullptr;
        check(mw_predictor_create(&q) == MW_OK, "launch-shape predictor create", shape);
        const int hkv = hkvs[uniform(0, 3)], group = uniform(1, 16);
        check(mw_predictor_set_launch_shape(q, hkv * group, hkv) == MW_OK, "set launch shape", shape);
        for (int it = 0; it < 60; ++it) {
            const int cus = 8 * uniform(1, 32), batch = uniform(1, 6);
            std::vector<int32_t> n(batch), r(batch);
            for (int b = 0; b < batch; ++b) {
                n[b] = uniform(1, 6000);
                r[b] = uniform(0, 70000);
            }
            mw_predictor_add_prefill(q, cus, batch, n.data(), r.data(), 0.01 + uniform(0, 100000) * 1e-4);
            if (it % 20 == 19) {
                mw_predictor_fit(q);
                double out = 0.0, th[4];
                if (mw_predictor_prefill_ms(q, cus, batch, n.data(), r.data(), &out) == MW_OK)
                    check(out == out && out < 1e30 && out > -1e30, "launch-shape prediction finite", it);
                mw_predictor_coefficients(q, 2 * uniform(0, 1), cus, th);
            }
        }
        mw_predictor_destroy(q);
    }
}

}  // namespace

int main() {
    planners();
    allocator();
    estimator();
    if (g_fail) return 1;
    std::printf("ok\n");
    return 0;
}
