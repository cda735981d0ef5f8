// Host tile-schedule builder and error reporting of libtriattn.so.
//
// The schedule lists, for every q-tile, the k-tiles the forward pass visits
// (Appendix A.1: sink blocks, then the sliding-window blocks of each
// streaming q-tile; the Last rows chunked over the whole key range).  It is
// computed in closed form from (cu_seqlens, sink, window, last, tile) with
// integer arithmetic only, so no block-index estimation happens at run time
// (Sec. 2.4: the pattern is static).
#include <algorithm>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "triattn_internal.h"

namespace triattn {

namespace {
thread_local std::string g_last_error;
}

ta_status fail(ta_status st, const char *fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    std::vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return st;
}

void clear_error() { g_last_error.clear(); }

namespace {

struct Item {
    int32_t w[kItemWords];
};
struct Merge {
    int32_t w[kMergeWords];
};

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

}  // namespace
}  // namespace triattn

using namespace triattn;

namespace {

// Write the packed schedule (header, split items, direct items, merges).
void pack_schedule(int32_t *w, int32_t kind, int32_t tile, int32_t batch, int32_t sink,
                   int32_t window, int32_t last, int32_t splits, int64_t total,
                   const std::vector<Item> &split_items, const std::vector<Item> &items,
                   const std::vector<Merge> &merges, int64_t partial_rows, int64_t kept,
                   int64_t merged_rows)
{
    w[H_MAGIC] = TA_SCHEDULE_MAGIC;
    w[H_VERSION] = TA_SCHEDULE_VERSION;
    w[H_KIND] = kind;
    w[H_TILE] = tile;
    w[H_BATCH] = batch;
    w[H_SINK] = sink;
    w[H_WINDOW] = window;
    w[H_LAST] = last;
    w[H_SPLITS] = splits;
    w[H_TOTAL_LO] = (int32_t)(uint32_t)((uint64_t)total & 0xffffffffu);
    w[H_TOTAL_HI] = (int32_t)(uint32_t)((uint64_t)total >> 32);
    w[H_ITEMS] = (int32_t)(split_items.size() + items.size());
    w[H_MERGES] = (int32_t)merges.size();
    w[H_PARTIAL_ROWS] = (int32_t)partial_rows;
    w[H_KEPT_TILES] = (int32_t)kept;
    w[H_LAST_ROWS] = (int32_t)merged_rows;
    w += kHdrWords;
    for (const Item &it : split_items) {
        std::memcpy(w, it.w, sizeof it.w);
        w += kItemWords;
    }
    for (const Item &it : items) {
        std::memcpy(w, it.w, sizeof it.w);
        w += kItemWords;
    }
    for (const Merge &m : merges) {
        std::memcpy(w, m.w, sizeof m.w);
        w += kMergeWords;
    }
}

constexpr int32_t kBlockSparseAutoTiles = 16;  // least automatic work bound

}  // namespace

extern "C" int32_t ta_abi_version(void) { return TA_ABI_VERSION; }

extern "C" const char *ta_last_error(void) { return g_last_error.c_str(); }

extern "C" ta_status ta_build_schedule(int32_t kind, const int32_t *cu_seqlens,
                                       int32_t batch, int32_t sink,
                                       int32_t window, int32_t last,
                                       int32_t tile, int32_t splits,
                                       int32_t *out, int64_t out_words,
                                       ta_schedule_info *info)
{
    clear_error();
    if (!info)
        return fail(TA_ERR_INVALID_ARG, "ta_build_schedule: info is NULL");
    if (kind != TA_KIND_TRIANGLE && kind != TA_KIND_CAUSAL)
        return fail(TA_ERR_INVALID_ARG, "ta_build_schedule: bad kind %d", kind);
    if (!cu_seqlens)
        return fail(TA_ERR_INVALID_ARG, "ta_build_schedule: cu_seqlens is NULL");
    if (batch < 0)
        return fail(TA_ERR_INVALID_ARG, "ta_build_schedule: batch %d < 0", batch);
    if (sink < 0 || window < 1 || last < 0 || splits < 0)
        return fail(TA_ERR_INVALID_ARG,
                    "ta_build_schedule: need sink >= 0, window >= 1, last >= 0,"
                    " splits >= 0 (got %d, %d, %d, %d)",
                    sink, window, last, splits);
    if (tile != 64 && tile != 128)
        return fail(TA_ERR_UNSUPPORTED, "ta_build_schedule: tile %d not in {64, 128}",
                    tile);
    if (out_words < 0)
        return fail(TA_ERR_INVALID_ARG, "ta_build_schedule: out_words < 0");
    if (cu_seqlens[0] != 0)
        return fail(TA_ERR_INVALID_ARG, "ta_build_schedule: cu_seqlens[0] != 0");
    for (int32_t b = 0; b < batch; ++b)
        if (cu_seqlens[b + 1] < cu_seqlens[b])
            return fail(TA_ERR_INVALID_ARG,
                        "ta_build_schedule: cu_seqlens decreases at %d", b);

    const int64_t T = tile;
    // Steady-state streaming work of one q-tile in k-tiles; the automatic
    // rule sizes Last splits to about that much work each, but to no fewer
    // than 2048 keys (32 steps of 64 keys), so that a split's fixed costs
    // (workgroup set-up, its partial rows and their merge) stay small
    // against its steps when the window is short.
    const int64_t t_star =
        std::max(ceil_div(sink, T) + ceil_div(window, T) + 1, ceil_div(2048, T));

    std::vector<Item> last_items, items;
    std::vector<Merge> merges;
    int64_t partial_rows = 0, kept = 0, last_rows_total = 0, max_splits = 0;
    int64_t max_item = 0;

    for (int32_t b = 0; b < batch; ++b) {
        const int64_t off = cu_seqlens[b];
        const int64_t n = cu_seqlens[b + 1] - off;
        if (n == 0)
            continue;
        const int64_t lr = kind == TA_KIND_TRIANGLE ? std::min<int64_t>(last, n) : 0;
        const int64_t split_row = n - lr;  // first Last row

        // Streaming q-tiles (or every q-tile of a causal pass).
        for (int64_t r0 = 0; r0 < split_row; r0 += T) {
            const int64_t r1 = std::min(r0 + T, split_row);
            int64_t ka0, ka1, kb0 = 0, kb1 = 0;
            if (kind == TA_KIND_CAUSAL) {
                ka0 = 0;
                ka1 = (r1 - 1) / T + 1;
            } else {
                // keys [0, min(sink, r1)) and [max(0, r0 - window + 1), r1 - 1]
                const int64_t sink_hi = ceil_div(std::min<int64_t>(sink, r1), T);
                const int64_t band_lo = std::max<int64_t>(0, r0 - window + 1) / T;
                const int64_t band_hi = (r1 - 1) / T + 1;
                if (sink_hi == 0) {
                    ka0 = band_lo;
                    ka1 = band_hi;
                } else if (band_lo <= sink_hi) {
                    ka0 = 0;
                    ka1 = std::max(sink_hi, band_hi);
                } else {
                    ka0 = 0;
                    ka1 = sink_hi;
                    kb0 = band_lo;
                    kb1 = band_hi;
                }
            }
            const int64_t cost = (ka1 - ka0) + (kb1 - kb0);
            kept += cost;
            max_item = std::max(max_item, cost);
            Item it = {{(int32_t)off, (int32_t)n, (int32_t)r0, (int32_t)r1,
                        (int32_t)ka0, (int32_t)ka1, (int32_t)kb0, (int32_t)kb1,
                        kind == TA_KIND_CAUSAL ? kModeCausal : kModeStreaming,
                        -1, (int32_t)cost, 0}};
            items.push_back(it);
        }

        // Last q-tiles: all k-tiles up to the diagonal, in balanced splits.
        for (int64_t r0 = split_row; r0 < n; r0 += T) {
            const int64_t r1 = std::min(r0 + T, n);
            const int64_t nk = (r1 - 1) / T + 1;
            int64_t ns = splits > 0 ? splits : ceil_div(nk, t_star);
            ns = std::max<int64_t>(1, std::min(ns, nk));
            kept += nk;
            for (int64_t c = 0; c < ns; ++c) {
                const int64_t k0 = c * nk / ns, k1 = (c + 1) * nk / ns;
                max_item = std::max(max_item, k1 - k0);
                Item it = {{(int32_t)off, (int32_t)n, (int32_t)r0, (int32_t)r1,
                            (int32_t)k0, (int32_t)k1, 0, 0, kModeCausal,
                            (int32_t)(partial_rows + c * (r1 - r0)),
                            (int32_t)(k1 - k0), 0}};
                last_items.push_back(it);
            }
            Merge m = {{(int32_t)off, (int32_t)r0, (int32_t)r1, (int32_t)ns,
                        (int32_t)partial_rows, 0, 0, 0}};
            merges.push_back(m);
            partial_rows += ns * (r1 - r0);
            last_rows_total += r1 - r0;
            max_splits = std::max(max_splits, ns);
            if (partial_rows > INT32_MAX)
                return fail(TA_ERR_UNSUPPORTED,
                            "ta_build_schedule: too many partial rows");
        }
    }

    if (kind == TA_KIND_CAUSAL)  // heaviest q-tiles first
        std::stable_sort(items.begin(), items.end(),
                         [](const Item &a, const Item &b) {
                             return a.w[I_COST] > b.w[I_COST];
                         });

    const int64_t n_main = (int64_t)last_items.size() + (int64_t)items.size();
    const int64_t words = kHdrWords + n_main * kItemWords +
                          (int64_t)merges.size() * kMergeWords;
    if (n_main > INT32_MAX / 64 || kept > INT32_MAX)
        return fail(TA_ERR_UNSUPPORTED, "ta_build_schedule: schedule too large");

    const int64_t total = cu_seqlens[batch];
    std::memset(info, 0, sizeof *info);
    info->version = TA_SCHEDULE_VERSION;
    info->kind = kind;
    info->tile = tile;
    info->batch = batch;
    info->sink = sink;
    info->window = window;
    info->last = last;
    info->splits_requested = splits;
    info->total_tokens = total;
    info->words = words;
    info->n_items = (int32_t)n_main;
    info->n_last_items = (int32_t)last_items.size();
    info->n_merge_items = (int32_t)merges.size();
    info->n_last_rows = (int32_t)last_rows_total;
    info->n_partial_rows = (int32_t)partial_rows;
    info->max_splits = (int32_t)max_splits;
    info->kept_tiles_per_qhead = kept;
    info->max_item_tiles = (int32_t)max_item;

    if (!out)
        return TA_OK;
    if (out_words < words)
        return fail(TA_ERR_BUFFER_TOO_SMALL,
                    "ta_build_schedule: out has %lld words, needs %lld",
                    (long long)out_words, (long long)words);

    pack_schedule(out, kind, tile, batch, sink, window, last, splits, total, last_items,
                  items, merges, partial_rows, kept, last_rows_total);
    return TA_OK;
}


extern "C" ta_status ta_build_blocksparse_schedule(const int32_t *cu_seqlens,
                                                   int32_t batch, int32_t tile,
                                                   const int32_t *qtile_ptr,
                                                   const int32_t *ktile_idx,
                                                   int32_t max_tiles_per_item,
                                                   int32_t *out, int64_t out_words,
                                                   ta_schedule_info *info)
{
    clear_error();
    static const char fn[] = "ta_build_blocksparse_schedule";
    if (!info)
        return fail(TA_ERR_INVALID_ARG, "%s: info is NULL", fn);
    if (!cu_seqlens || !qtile_ptr)
        return fail(TA_ERR_INVALID_ARG, "%s: cu_seqlens or qtile_ptr is NULL", fn);
    if (batch < 0 || max_tiles_per_item < 0 || out_words < 0)
        return fail(TA_ERR_INVALID_ARG,
                    "%s: need batch >= 0, max_tiles_per_item >= 0, out_words >= 0", fn);
    if (tile != 64 && tile != 128)
        return fail(TA_ERR_UNSUPPORTED, "%s: tile %d not in {64, 128}", fn, tile);
    if (cu_seqlens[0] != 0)
        return fail(TA_ERR_INVALID_ARG, "%s: cu_seqlens[0] != 0", fn);
    for (int32_t b = 0; b < batch; ++b)
        if (cu_seqlens[b + 1] < cu_seqlens[b])
            return fail(TA_ERR_INVALID_ARG, "%s: cu_seqlens decreases at %d", fn, b);
    if (qtile_ptr[0] != 0)
        return fail(TA_ERR_INVALID_ARG, "%s: qtile_ptr[0] != 0", fn);

    const int64_t T = tile;
    // Automatic bound: only q-tiles listing more than twice the mean number
    // of tiles are cut (and never into chunks under 16 tiles), so uniform
    // lists stay whole and a skewed list does not set the critical path.
    int64_t n_qtiles = 0;
    for (int32_t b = 0; b < batch; ++b)
        n_qtiles += ceil_div((int64_t)cu_seqlens[b + 1] - cu_seqlens[b], T);
    const int64_t listed = std::max<int64_t>(0, qtile_ptr[n_qtiles]);
    const int64_t M = max_tiles_per_item > 0
                          ? max_tiles_per_item
                          : std::max<int64_t>(kBlockSparseAutoTiles,
                                              ceil_div(2 * listed, std::max<int64_t>(n_qtiles, 1)));
    std::vector<Item> split_items, items;
    std::vector<Merge> merges;
    int64_t partial_rows = 0, merged_rows = 0, max_splits = 0, max_item = 0;
    int64_t qt = 0;  // global q-tile index

    for (int32_t b = 0; b < batch; ++b) {
        const int64_t off = cu_seqlens[b];
        const int64_t n = cu_seqlens[b + 1] - off;
        for (int64_t t = 0; t * T < n; ++t, ++qt) {
            const int64_t p0 = qtile_ptr[qt], p1 = qtile_ptr[qt + 1];
            if (p1 < p0)
                return fail(TA_ERR_INVALID_ARG, "%s: qtile_ptr decreases at q-tile %lld",
                            fn, (long long)qt);
            if (p1 > p0 && !ktile_idx)
                return fail(TA_ERR_INVALID_ARG, "%s: ktile_idx is NULL", fn);
            for (int64_t p = p0; p < p1; ++p) {
                const int64_t kt = ktile_idx[p];
                if (kt < 0 || kt > t || (p > p0 && kt <= ktile_idx[p - 1]))
                    return fail(TA_ERR_INVALID_ARG,
                                "%s: q-tile %lld: k-tile %lld out of order or above the "
                                "diagonal", fn, (long long)qt, (long long)kt);
            }
            if (p1 > INT32_MAX)
                return fail(TA_ERR_UNSUPPORTED, "%s: lists too long", fn);
            const int64_t r0 = t * T, r1 = std::min(r0 + T, n);
            // balanced chunks of the list, at most M tiles each, in order
            const int64_t len = p1 - p0;
            const int64_t ns = std::max<int64_t>(1, ceil_div(len, M));
            std::vector<Item> q_items;
            for (int64_t c = 0; c < ns; ++c) {
                const int64_t a = c * len / ns, z = (c + 1) * len / ns;
                max_item = std::max(max_item, z - a);
                Item it = {{(int32_t)off, (int32_t)n, (int32_t)r0, (int32_t)r1,
                            (int32_t)(p0 + a), (int32_t)(z - a), 0, 0, kModeCausalList,
                            -1, (int32_t)(z - a), 0}};
                q_items.push_back(it);
            }
            if (ns == 1) {
                items.push_back(q_items[0]);
                continue;
            }
            for (int64_t c = 0; c < ns; ++c) {
                q_items[c].w[I_PART_BASE] = (int32_t)(partial_rows + c * (r1 - r0));
                split_items.push_back(q_items[c]);
            }
            Merge m = {{(int32_t)off, (int32_t)r0, (int32_t)r1, (int32_t)ns,
                        (int32_t)partial_rows, 0, 0, 0}};
            merges.push_back(m);
            partial_rows += ns * (r1 - r0);
            merged_rows += r1 - r0;
            max_splits = std::max(max_splits, ns);
            if (partial_rows > INT32_MAX)
                return fail(TA_ERR_UNSUPPORTED, "%s: too many partial rows", fn);
        }
    }
    const int64_t list_words = qtile_ptr[qt];
    auto by_cost = [](const Item &a, const Item &b) { return a.w[I_COST] > b.w[I_COST]; };
    std::stable_sort(split_items.begin(), split_items.end(), by_cost);
    std::stable_sort(items.begin(), items.end(), by_cost);

    const int64_t n_main = (int64_t)split_items.size() + (int64_t)items.size();
    const int64_t words = kHdrWords + n_main * kItemWords +
                          (int64_t)merges.size() * kMergeWords + list_words;
    if (n_main > INT32_MAX / 64 || list_words > INT32_MAX / 2)
        return fail(TA_ERR_UNSUPPORTED, "%s: schedule too large", fn);
    const int64_t total = cu_seqlens[batch];
    std::memset(info, 0, sizeof *info);
    info->version = TA_SCHEDULE_VERSION;
    info->kind = TA_KIND_BLOCKSPARSE;
    info->tile = tile;
    info->batch = batch;
    info->window = (int32_t)list_words;
    info->splits_requested = max_tiles_per_item;
    info->total_tokens = total;
    info->words = words;
    info->n_items = (int32_t)n_main;
    info->n_last_items = (int32_t)split_items.size();
    info->n_merge_items = (int32_t)merges.size();
    info->n_last_rows = (int32_t)merged_rows;
    info->n_partial_rows = (int32_t)partial_rows;
    info->max_splits = (int32_t)max_splits;
    info->kept_tiles_per_qhead = list_words;
    info->max_item_tiles = (int32_t)max_item;
    if (!out)
        return TA_OK;
    if (out_words < words)
        return fail(TA_ERR_BUFFER_TOO_SMALL, "%s: out has %lld words, needs %lld", fn,
                    (long long)out_words, (long long)words);
    pack_schedule(out, TA_KIND_BLOCKSPARSE, tile, batch, 0, (int32_t)list_words, 0,
                  max_tiles_per_item, total, split_items, items, merges, partial_rows,
                  list_words, merged_rows);
    if (list_words > 0)
        std::memcpy(out + (words - list_words), ktile_idx, sizeof(int32_t) * list_words);
    return TA_OK;
}

extern "C" size_t ta_workspace_bytes(const ta_schedule_info *info, int32_t hq,
                                     int32_t head_dim)
{
    if (!info || hq <= 0 || head_dim <= 0 || info->n_partial_rows <= 0)
        return 0;
    const size_t rows = (size_t)info->n_partial_rows * (size_t)hq;
    const size_t o_bytes = (rows * (size_t)head_dim * 4 + 255) & ~(size_t)255;
    const size_t l_bytes = (rows * 4 + 255) & ~(size_t)255;
    return o_bytes + l_bytes;
}
