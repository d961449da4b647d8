// Internal declarations shared by the library's translation units.
#pragma once

#include <hip/hip_runtime.h>

#include <chrono>
#include <cstdint>
#include <deque>
#include <vector>

#include "mw.h"

namespace mw {

constexpr int kHeadDim = 128;
constexpr int kPageSize = 16;
constexpr int kMaxTimingEvents = 8;

// Records `msg` as the calling thread's last error and returns `st`.
mw_status fail(mw_status st, const char *fmt, ...) __attribute__((format(printf, 2, 3)));

inline bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Key-range split of the prefill query blocks of the 4-wave kernel: a block
// whose causal key range spans nt tiles of 64 keys is cut into this many
// pieces, piece i covering tiles [i nt / k, (i + 1) nt / k).  With
// piece_tiles >= 4 every cut lies at least two tiles before the block's end,
// so the first tile of every piece holds a key that every query of the block
// sees (a block's last two tiles hold its diagonal).
constexpr int kPrefillMaxPieces = 8;
constexpr int kPrefillMinPieceTiles = 4;
__host__ __device__ inline int prefill_pieces(int nt, int piece_tiles, int max_pieces) {
    const int k = (nt + piece_tiles - 1) / piece_tiles;
    return k < 1 ? 1 : (k > max_pieces ? max_pieces : k);
}
// Key tiles (64 keys) of the 32-position query block q of a sequence with
// prefix r and n new tokens.
__host__ __device__ inline int prefill_block_tiles(int r, int n, int q) {
    const int end = 32 * q + 32 < n ? 32 * q + 32 : n;
    return (r + end + 63) / 64;
}

// Number of CUs a stream's kernels may run on (its CU mask; all CUs of the
// current device for a stream without one).
int stream_cus(hipStream_t s);

}  // namespace mw

#define MW_HIP_TRY(expr)                                                                  \
    do {                                                                                  \
        hipError_t mw_e_ = (expr);                                                        \
        if (mw_e_ != hipSuccess)                                                          \
            return mw::fail(MW_ERR_HIP, "%s failed: %s", #expr, hipGetErrorString(mw_e_)); \
    } while (0)

struct mw_kv_pool {
    mw_kv_pool_desc desc;
    uint16_t *k;
    uint16_t *v;
    std::deque<int32_t> free_list;
    std::vector<uint8_t> is_free;
};

struct mw_timing {
    hipEvent_t ev[mw::kMaxTimingEvents];
    int n_events;          // events recorded by the last call (start + one per kernel)
    bool created;
    double host_ms;        // host time spent enqueueing
    std::chrono::steady_clock::time_point t0;
};

struct mw_partition {
    int device;
    hipStream_t prefill;
    hipStream_t decode;
    uint32_t prefill_mask[8];
    uint32_t decode_mask[8];
};

namespace mw {

// Timing helpers: begin() records the start event, kernel_done() one event per
// kernel, end() the host-side duration.  All are no-ops for a NULL handle.
mw_status timing_begin(mw_timing *t, hipStream_t s);
mw_status timing_kernel_done(mw_timing *t, hipStream_t s);
void timing_end(mw_timing *t);

// Reports a failed kernel launch (bad configuration) as MW_ERR_HIP.
mw_status check_launch(const char *what);

}  // namespace mw

namespace mw {

// Checked launch parameters of one decode call (shared by mw_decode_attn and
// the fused kernel's launcher).
struct DecodePlan {
    int64_t units;        // work-groups of the split kernel
    int chunk_pages;      // fixed chunks: resolved chunk length; 0 with the balanced split
    int64_t per_unit;     // balanced split: pages per unit (0 with fixed chunks)
    int64_t total;        // balanced split: pages of all (sequence, kv head) segments, in the split's numbering
    bool aligned;         // balanced split: each segment padded to a multiple of per_unit pages
    int64_t slots;        // partial slots in the workspace
    // workspace layout: partial O, (m, l), then per-sequence chunk bases (fixed
    // chunks) or per-slot done flags (balanced split)
    size_t off_ml, off_meta, bytes;
    int hkv, group;
    float scale_log2;
};
// Validates a decode call's arguments (workspace size included) and plans it.
// cus > 0 with chunk_pages = 0: the balanced split over that many CUs;
// cus = 0: fixed chunks only (chunk_pages 0 then means automatic chunks).
mw_status decode_prepare(const mw_decode_args *a, int64_t cus, DecodePlan *p, const char *who);
// Launches the kernel that merges the chunk partials of every (sequence, kv
// head) of a fixed-chunk split (the balanced split merges its own).
mw_status decode_combine_launch(const mw_decode_args *a, const DecodePlan &p, hipStream_t s);

// Checked launch parameters of one prefill call.
struct PrefillPlan {
    int hkv, group, n_hgroups, paired;
    int waves;            // 8 (64-position query blocks) or 4 (32-position blocks)
    int64_t gx;           // work-groups per sequence (grid x); 0: nothing to do
    int batch;
    bool table_in_lds;    // every block-table entry a work-group needs fits its LDS copy
    float scale_log2;
    // key-range split (4-wave blocks only; planned by prefill_split_plan)
    int pieces;           // most pieces of any block; 1: no split
    int piece_tiles;      // target key tiles per piece
    int64_t rows;         // sum of the new lengths (rows of the workspace partials)
    size_t split_bytes;   // workspace the split needs
};
// Validates a prefill call's arguments and plans it for a stream that may use
// `cus` CUs (block pairing and, with allow_small, the work-group size depend
// on it).
mw_status prefill_prepare(const mw_prefill_args *a, int64_t cus, bool allow_small, PrefillPlan *p, const char *who);
// The launch plan of a prefill call from its lengths alone (no validation):
// waves, pairing and grid width for a stream of `cus` CUs; used by
// prefill_prepare and by the latency predictor, which simulates the launch.
void prefill_plan_lengths(int32_t batch, const int32_t *h_new_lens, int hkv, int group, int64_t cus,
                          bool allow_small, PrefillPlan *p);
// Plans the key-range split of a 4-wave call on `cus` CUs (cus = 0: the
// largest split any stream could take); fills pieces, piece_tiles, rows and
// split_bytes.  Lengths must have been validated.
void prefill_split_plan(int32_t batch, const int32_t *h_new_lens, const int32_t *h_prefix_lens, int hq,
                        int64_t cus, PrefillPlan *p);

}  // namespace mw
