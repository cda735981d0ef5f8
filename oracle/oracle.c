/*
 * oracle.c -- plain, slow, fp64 CPU reference for Triangle attention and
 * dense causal attention (arXiv 2507.21526).
 *
 * TEST INFRASTRUCTURE ONLY: used by the tests, the smoke check and the CPU
 * baseline of the benchmark; never by the product path.  It shares no code
 * with the HIP library: the masks are evaluated element by element from the
 * region definitions of Appendix A.3, attention is the masked softmax of
 * Sec. 2.1 evaluated row by row in double precision, and the tile schedule is
 * found by brute force over every (q-tile, k-tile) block.
 */
#include "oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

static double widen_bf16(uint16_t bits)
{
    uint32_t u = (uint32_t)bits << 16; /* bf16 is the top half of an fp32 */
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

/* ---- Appendix A.3: the three sections of the causal attention matrix ---- */

/* Streaming section: the sink keys and the sliding window, causal. */
int oracle_in_streaming(int64_t i, int64_t j, int64_t sink, int64_t window)
{
    if (!(i >= j))
        return 0;
    return (j < sink) || (i - j < window);
}

static int64_t last_rows(int64_t n, int64_t last)
{
    return last < n ? last : n;
}

/* Last Q-K section: the last rows, outside the streaming section, causal. */
int oracle_in_last(int64_t i, int64_t j, int64_t n, int64_t sink,
                   int64_t window, int64_t last)
{
    if (!(i >= j))
        return 0;
    if (!(i >= n - last_rows(n, last)))
        return 0;
    return (j >= sink) && (i - j >= window);
}

/* Middle Q-K section: what Triangle attention skips. */
int oracle_in_middle(int64_t i, int64_t j, int64_t n, int64_t sink,
                     int64_t window, int64_t last)
{
    if (!(i >= j))
        return 0;
    if (!(i < n - last_rows(n, last)))
        return 0;
    return (j >= sink) && (i - j >= window);
}

/* Sec. 2.4: Triangle = Streaming section plus Last Q-K section. */
int oracle_mask(int kind, int64_t i, int64_t j, int64_t n, int64_t sink,
                int64_t window, int64_t last)
{
    if (kind == ORACLE_CAUSAL)
        return i >= j;
    return oracle_in_streaming(i, j, sink, window) ||
           oracle_in_last(i, j, n, sink, window, last);
}

void oracle_mask_row(int kind, int64_t n, int64_t sink, int64_t window,
                     int64_t last, int64_t i, uint8_t *row)
{
    for (int64_t j = 0; j < n; ++j)
        row[j] = (uint8_t)oracle_mask(kind, i, j, n, sink, window, last);
}

int64_t oracle_mask_nnz(int kind, int64_t n, int64_t sink, int64_t window,
                        int64_t last)
{
    int64_t total = 0;
#pragma omp parallel for reduction(+ : total) schedule(dynamic, 64)
    for (int64_t i = 0; i < n; ++i)
        for (int64_t j = 0; j < n; ++j)
            total += oracle_mask(kind, i, j, n, sink, window, last);
    return total;
}

/* ---- Sec. 2.1: masked softmax attention, one (row, head) at a time ---- */

/* Mask row source: fills row[0..n) for row i of sequence b. */
typedef struct {
    int kind;
    int64_t sink, window, last;
    /* block-sparse lists (kind < 0) */
    int64_t tile;
    const int32_t *qtile_ptr, *ktile_idx, *qbase;
} mask_src;

static void fill_mask_row(const mask_src *ms, int32_t b, int64_t n, int64_t i,
                          uint8_t *row)
{
    if (ms->kind >= 0) {
        oracle_mask_row(ms->kind, n, ms->sink, ms->window, ms->last, i, row);
        return;
    }
    const int64_t g = ms->qbase[b] + i / ms->tile;
    const int32_t *list = ms->ktile_idx + ms->qtile_ptr[g];
    const int64_t len = ms->qtile_ptr[g + 1] - ms->qtile_ptr[g];
    for (int64_t j = 0; j < n; ++j)
        row[j] = (uint8_t)oracle_bs_mask(i, j, ms->tile, list, len);
}

/* Masked softmax attention of the requested rows (Sec. 2.1). */
static int attn_rows_core(const uint16_t *q, const uint16_t *k, const uint16_t *v,
                          const int32_t *cu_seqlens, int32_t batch, int32_t hq,
                          int32_t hkv, int32_t d, const mask_src *ms,
                          double scale, const int64_t *row_tok,
                          const int32_t *row_head, int64_t nrows, double *out,
                          double *lse, double *absw)
{
    if (batch < 0 || hq <= 0 || hkv <= 0 || d <= 0 || hq % hkv != 0)
        return -1;
    const int64_t total = cu_seqlens[batch];
    const int32_t group = hq / hkv;
    for (int64_t r = 0; r < nrows; ++r) {
        if (row_tok[r] < 0 || row_tok[r] >= total || row_head[r] < 0 ||
            row_head[r] >= hq)
            return -1;
    }

    int bad = 0;
#pragma omp parallel
    {
        int64_t cap = 0;
        uint8_t *mask = NULL;
        double *z = NULL;
#pragma omp for schedule(dynamic, 1)
        for (int64_t r = 0; r < nrows; ++r) {
            const int64_t t = row_tok[r];
            const int32_t h = row_head[r];
            const int32_t g = h / group;
            int32_t b = 0;
            while (!(cu_seqlens[b] <= t && t < cu_seqlens[b + 1]))
                ++b;
            const int64_t off = cu_seqlens[b];
            const int64_t n = cu_seqlens[b + 1] - off;
            const int64_t i = t - off;
            if (n > cap) {
                free(mask);
                free(z);
                cap = n;
                mask = (uint8_t *)malloc((size_t)n);
                z = (double *)malloc((size_t)n * sizeof(double));
            }
            if (!mask || !z) {
#pragma omp atomic write
                bad = 1;
                continue;
            }
            fill_mask_row(ms, b, n, i, mask);

            const uint16_t *qi = q + ((size_t)t * hq + h) * d;
            double zmax = -INFINITY;
            for (int64_t j = 0; j < n; ++j) {
                if (!mask[j])
                    continue;
                const uint16_t *kj = k + ((size_t)(off + j) * hkv + g) * d;
                double dot = 0.0;
                for (int32_t c = 0; c < d; ++c)
                    dot += widen_bf16(qi[c]) * widen_bf16(kj[c]);
                z[j] = scale * dot;
                if (z[j] > zmax)
                    zmax = z[j];
            }
            double *o = out + (size_t)r * d;
            double *aw = absw ? absw + (size_t)r * d : NULL;
            for (int32_t c = 0; c < d; ++c)
                o[c] = 0.0;
            if (aw)
                for (int32_t c = 0; c < d; ++c)
                    aw[c] = 0.0;
            double denom = 0.0;
            for (int64_t j = 0; j < n; ++j) {
                if (!mask[j])
                    continue;
                const double p = exp(z[j] - zmax);
                denom += p;
                const uint16_t *vj = v + ((size_t)(off + j) * hkv + g) * d;
                for (int32_t c = 0; c < d; ++c)
                    o[c] += p * widen_bf16(vj[c]);
                if (aw)
                    for (int32_t c = 0; c < d; ++c)
                        aw[c] += p * fabs(widen_bf16(vj[c]));
            }
            if (denom > 0.0) {
                for (int32_t c = 0; c < d; ++c)
                    o[c] /= denom;
                if (aw)
                    for (int32_t c = 0; c < d; ++c)
                        aw[c] /= denom;
            }
            if (lse)
                lse[r] = denom > 0.0 ? zmax + log(denom) : -INFINITY;
        }
        free(mask);
        free(z);
    }
    return bad ? -1 : 0;
}

int oracle_attn_rows(const uint16_t *q, const uint16_t *k, const uint16_t *v,
                     const int32_t *cu_seqlens, int32_t batch, int32_t hq,
                     int32_t hkv, int32_t d, int kind, int64_t sink,
                     int64_t window, int64_t last, double scale,
                     const int64_t *row_tok, const int32_t *row_head,
                     int64_t nrows, double *out, double *lse)
{
    if (kind != ORACLE_TRIANGLE && kind != ORACLE_CAUSAL)
        return -1;
    mask_src ms = {kind, sink, window, last, 0, NULL, NULL, NULL};
    return attn_rows_core(q, k, v, cu_seqlens, batch, hq, hkv, d, &ms, scale,
                          row_tok, row_head, nrows, out, lse, NULL);
}

int oracle_attn_rows_absw(const uint16_t *q, const uint16_t *k, const uint16_t *v,
                          const int32_t *cu_seqlens, int32_t batch, int32_t hq,
                          int32_t hkv, int32_t d, int kind, int64_t sink,
                          int64_t window, int64_t last, double scale,
                          const int64_t *row_tok, const int32_t *row_head,
                          int64_t nrows, double *out, double *lse, double *absw)
{
    if (kind != ORACLE_TRIANGLE && kind != ORACLE_CAUSAL)
        return -1;
    mask_src ms = {kind, sink, window, last, 0, NULL, NULL, NULL};
    return attn_rows_core(q, k, v, cu_seqlens, batch, hq, hkv, d, &ms, scale,
                          row_tok, row_head, nrows, out, lse, absw);
}

/* ---- Block-sparse causal attention ---- */

int oracle_bs_mask(int64_t i, int64_t j, int64_t tile, const int32_t *list,
                   int64_t len)
{
    if (j > i)
        return 0;
    const int64_t kt = j / tile;
    for (int64_t p = 0; p < len; ++p)
        if (list[p] == kt)
            return 1;
    return 0;
}

/* First global q-tile of each sequence; returns NULL on failure. */
static int32_t *qtile_bases(const int32_t *cu_seqlens, int32_t batch, int64_t tile)
{
    int32_t *base = (int32_t *)malloc(sizeof(int32_t) * (size_t)(batch + 1));
    if (!base)
        return NULL;
    int64_t acc = 0;
    for (int32_t b = 0; b < batch; ++b) {
        base[b] = (int32_t)acc;
        acc += (cu_seqlens[b + 1] - cu_seqlens[b] + tile - 1) / tile;
    }
    base[batch] = (int32_t)acc;
    return base;
}

int oracle_attn_rows_bs(const uint16_t *q, const uint16_t *k, const uint16_t *v,
                        const int32_t *cu_seqlens, int32_t batch, int32_t hq,
                        int32_t hkv, int32_t d, int32_t tile,
                        const int32_t *qtile_ptr, const int32_t *ktile_idx,
                        double scale, const int64_t *row_tok,
                        const int32_t *row_head, int64_t nrows, double *out,
                        double *lse)
{
    if (tile < 1 || batch < 0)
        return -1;
    int32_t *base = qtile_bases(cu_seqlens, batch, tile);
    if (!base)
        return -1;
    mask_src ms = {-1, 0, 0, 0, tile, qtile_ptr, ktile_idx, base};
    const int rc = attn_rows_core(q, k, v, cu_seqlens, batch, hq, hkv, d, &ms,
                                  scale, row_tok, row_head, nrows, out, lse, NULL);
    free(base);
    return rc;
}

/* ---- Tile schedule by brute force over blocks ----
 *
 * Packed int32 format (documented with the library's interface):
 *   header, 16 words: magic, version, kind, tile, batch, sink, window, last,
 *     splits requested, total_tokens (low, high 32 bits), main items, merge
 *     items, partial rows, kept k-tiles per query head, rows of the Last
 *     q-tiles (the rows the merge items cover).
 *   main item, 12 words: seq_off, seq_len, r0, r1, ka0, ka1, kb0, kb1, mode,
 *     part_base, kept k-tiles, 0.   Rows [r0, r1) are relative to the
 *     sequence start; [ka0, ka1) and [kb0, kb1) are the kept k-tiles as at
 *     most two maximal runs in increasing order (an absent run is (0, 0));
 *     mode 0 = streaming mask, 1 = causal mask, 2 = causal mask over the
 *     k-tiles lists[ka0 .. ka0 + ka1) of the list section (block-sparse);
 *     part_base -1 = the item writes the output rows, else it writes partial
 *     rows part_base + (i - r0).
 *   k-tile lists (block-sparse only): header word 6 words after the merges.
 *   merge item, 8 words: seq_off, r0, r1, splits, part_base, 0, 0, 0.
 * Triangle order: the Last split items (by sequence, q-tile, split), then the
 * streaming items (by sequence, q-tile).  Causal order: by kept k-tiles,
 * descending, ties in (sequence, q-tile) order.
 */

enum { HDR_WORDS = 16, ITEM_WORDS = 12, MERGE_WORDS = 8 };
static const int32_t SCHED_MAGIC = 0x54524941;
static const int32_t SCHED_VERSION = 2;

typedef struct {
    int32_t w[ITEM_WORDS];
} item_t;

typedef struct {
    item_t *v;
    int64_t n, cap;
} item_vec;

static int push_item(item_vec *iv, const item_t *it)
{
    if (iv->n == iv->cap) {
        int64_t nc = iv->cap ? 2 * iv->cap : 256;
        item_t *nv = (item_t *)realloc(iv->v, (size_t)nc * sizeof(item_t));
        if (!nv)
            return -1;
        iv->v = nv;
        iv->cap = nc;
    }
    iv->v[iv->n++] = *it;
    return 0;
}

static void stable_sort_by_cost(item_vec *iv)
{
    for (int64_t a = 1; a < iv->n; ++a) {
        item_t x = iv->v[a];
        int64_t p = a - 1;
        while (p >= 0 && iv->v[p].w[10] < x.w[10]) {
            iv->v[p + 1] = iv->v[p];
            --p;
        }
        iv->v[p + 1] = x;
    }
}

/* kept[qt * nkt + kt] = 1 iff block (q-tile qt, k-tile kt) holds a kept pair.
 * q-tile qt covers rows [row0 + qt*tile, min(row0 + (qt+1)*tile, row1)). */
static void kept_blocks(int kind, int64_t n, int64_t sink, int64_t window,
                        int64_t last, int64_t tile, int64_t row0,
                        int64_t row1, int64_t nqt, int64_t nkt, uint8_t *kept)
{
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t qt = 0; qt < nqt; ++qt) {
        const int64_t r0 = row0 + qt * tile;
        const int64_t r1 = (r0 + tile < row1) ? r0 + tile : row1;
        for (int64_t kt = 0; kt < nkt; ++kt) {
            const int64_t c0 = kt * tile;
            const int64_t c1 = (c0 + tile < n) ? c0 + tile : n;
            int any = 0;
            for (int64_t i = r0; i < r1 && !any; ++i)
                for (int64_t j = c0; j < c1; ++j)
                    any |= oracle_mask(kind, i, j, n, sink, window, last);
            kept[qt * nkt + kt] = (uint8_t)(any != 0);
        }
    }
}

/* Split maximal runs of kept k-tiles; returns the number of runs (<= 2 kept). */
static int runs_of(const uint8_t *kept, int64_t nkt, int64_t run[2][2])
{
    int nruns = 0;
    run[0][0] = run[0][1] = run[1][0] = run[1][1] = 0;
    for (int64_t kt = 0; kt < nkt;) {
        if (!kept[kt]) {
            ++kt;
            continue;
        }
        int64_t e = kt;
        while (e < nkt && kept[e])
            ++e;
        if (nruns >= 2)
            return 3;
        run[nruns][0] = kt;
        run[nruns][1] = e;
        ++nruns;
        kt = e;
    }
    return nruns;
}

int64_t oracle_schedule(int kind, const int32_t *cu_seqlens, int32_t batch,
                        int32_t sink, int32_t window, int32_t last,
                        int32_t tile, int32_t splits, int32_t *out,
                        int64_t cap)
{
    if ((kind != ORACLE_TRIANGLE && kind != ORACLE_CAUSAL) || batch < 0 ||
        tile < 1 || sink < 0 || window < 1 || last < 0 || splits < 0 ||
        cu_seqlens[0] != 0)
        return -1;
    for (int32_t b = 0; b < batch; ++b)
        if (cu_seqlens[b + 1] < cu_seqlens[b])
            return -1;

    item_vec last_items = {0}, main_items = {0}, merges = {0};
    int64_t partial_rows = 0, kept_total = 0, merged_rows = 0;
    int fail = 0;
    /* steady-state streaming work of one q-tile, in k-tiles, and at least
     * 2048 keys' worth (reading 8: Algorithm 1 leaves the split count open) */
    int64_t t_star = (sink + tile - 1) / tile + (window + tile - 1) / tile + 1;
    if (t_star < (2048 + tile - 1) / tile)
        t_star = (2048 + tile - 1) / tile;

    for (int32_t b = 0; b < batch && !fail; ++b) {
        const int64_t off = cu_seqlens[b];
        const int64_t n = cu_seqlens[b + 1] - off;
        if (n == 0)
            continue;
        const int64_t nkt = (n + tile - 1) / tile;
        const int64_t lr = (kind == ORACLE_TRIANGLE) ? last_rows(n, last) : 0;
        /* region 0: rows [0, n - lr) ; region 1 (Triangle only): [n - lr, n) */
        for (int region = 0; region < 2 && !fail; ++region) {
            const int64_t row0 = region == 0 ? 0 : n - lr;
            const int64_t row1 = region == 0 ? n - lr : n;
            if (row1 <= row0)
                continue;
            const int64_t nqt = (row1 - row0 + tile - 1) / tile;
            uint8_t *kept = (uint8_t *)malloc((size_t)(nqt * nkt));
            if (!kept) {
                fail = 1;
                break;
            }
            kept_blocks(kind, n, sink, window, last, tile, row0, row1, nqt,
                        nkt, kept);
            for (int64_t qt = 0; qt < nqt && !fail; ++qt) {
                const int64_t r0 = row0 + qt * tile;
                const int64_t r1 = (r0 + tile < row1) ? r0 + tile : row1;
                int64_t run[2][2];
                const int nr = runs_of(kept + qt * nkt, nkt, run);
                if (nr < 1 || nr > 2) {
                    fail = 1;
                    break;
                }
                const int64_t cost = (run[0][1] - run[0][0]) +
                                     (run[1][1] - run[1][0]);
                kept_total += cost;
                if (region == 0) {
                    item_t it = {{(int32_t)off, (int32_t)n, (int32_t)r0,
                                  (int32_t)r1, (int32_t)run[0][0],
                                  (int32_t)run[0][1], (int32_t)run[1][0],
                                  (int32_t)run[1][1],
                                  kind == ORACLE_CAUSAL ? 1 : 0, -1,
                                  (int32_t)cost, 0}};
                    fail |= push_item(&main_items, &it);
                    continue;
                }
                /* Last q-tile: every k-tile up to the diagonal, cut into
                 * balanced contiguous splits (Appendix A.1, Alg. 1). */
                if (nr != 1 || run[0][0] != 0) {
                    fail = 1;
                    break;
                }
                const int64_t nk = run[0][1];
                int64_t ns = splits > 0 ? splits : (nk + t_star - 1) / t_star;
                if (ns < 1)
                    ns = 1;
                if (ns > nk)
                    ns = nk;
                for (int64_t c = 0; c < ns; ++c) {
                    const int64_t k0 = c * nk / ns, k1 = (c + 1) * nk / ns;
                    item_t it = {{(int32_t)off, (int32_t)n, (int32_t)r0,
                                  (int32_t)r1, (int32_t)k0, (int32_t)k1, 0, 0,
                                  1, (int32_t)(partial_rows + c * (r1 - r0)),
                                  (int32_t)(k1 - k0), 0}};
                    fail |= push_item(&last_items, &it);
                }
                item_t m = {{(int32_t)off, (int32_t)r0, (int32_t)r1,
                             (int32_t)ns, (int32_t)partial_rows, 0, 0, 0, 0,
                             0, 0, 0}};
                fail |= push_item(&merges, &m);
                partial_rows += ns * (r1 - r0);
                merged_rows += r1 - r0;
            }
            free(kept);
        }
    }

    if (!fail && kind == ORACLE_CAUSAL)
        /* stable ordering by kept k-tiles, descending (insertion sort keeps
         * equal costs in their (sequence, q-tile) order) */
        stable_sort_by_cost(&main_items);

    int64_t words = -1;
    if (!fail) {
        const int64_t n_main = last_items.n + main_items.n;
        words = HDR_WORDS + n_main * ITEM_WORDS + merges.n * MERGE_WORDS;
        if (out && cap >= words) {
            const int64_t total = cu_seqlens[batch];
            int32_t *w = out;
            w[0] = SCHED_MAGIC;
            w[1] = SCHED_VERSION;
            w[2] = kind;
            w[3] = tile;
            w[4] = batch;
            w[5] = sink;
            w[6] = window;
            w[7] = last;
            w[8] = splits;
            w[9] = (int32_t)(uint32_t)((uint64_t)total & 0xffffffffu);
            w[10] = (int32_t)(uint32_t)((uint64_t)total >> 32);
            w[11] = (int32_t)n_main;
            w[12] = (int32_t)merges.n;
            w[13] = (int32_t)partial_rows;
            w[14] = (int32_t)kept_total;
            w[15] = (int32_t)merged_rows;
            w += HDR_WORDS;
            for (int64_t a = 0; a < last_items.n; ++a, w += ITEM_WORDS)
                memcpy(w, last_items.v[a].w, sizeof(int32_t) * ITEM_WORDS);
            for (int64_t a = 0; a < main_items.n; ++a, w += ITEM_WORDS)
                memcpy(w, main_items.v[a].w, sizeof(int32_t) * ITEM_WORDS);
            for (int64_t a = 0; a < merges.n; ++a, w += MERGE_WORDS)
                memcpy(w, merges.v[a].w, sizeof(int32_t) * MERGE_WORDS);
        }
    }
    free(last_items.v);
    free(main_items.v);
    free(merges.v);
    return words;
}

int64_t oracle_bs_schedule(const int32_t *cu_seqlens, int32_t batch,
                           int32_t tile, const int32_t *qtile_ptr,
                           const int32_t *ktile_idx, int32_t max_tiles,
                           int32_t *out, int64_t cap)
{
    if (batch < 0 || tile < 1 || max_tiles < 0 || cu_seqlens[0] != 0 ||
        qtile_ptr[0] != 0)
        return -1;
    for (int32_t b = 0; b < batch; ++b)
        if (cu_seqlens[b + 1] < cu_seqlens[b])
            return -1;
    /* automatic bound: twice the mean list length over all q-tiles, at
     * least 16 */
    int64_t nq_all = 0;
    for (int32_t b = 0; b < batch; ++b)
        nq_all += (cu_seqlens[b + 1] - cu_seqlens[b] + tile - 1) / tile;
    int64_t bound = max_tiles;
    if (max_tiles == 0) {
        const int64_t listed = qtile_ptr[nq_all] > 0 ? qtile_ptr[nq_all] : 0;
        const int64_t nq = nq_all > 0 ? nq_all : 1;
        bound = (2 * listed + nq - 1) / nq;
        if (bound < 16)
            bound = 16;
    }
    item_vec split_items = {0}, items = {0}, merges = {0};
    int64_t partial_rows = 0, merged_rows = 0;
    int32_t *kept_list = NULL; /* concatenated kept k-tiles of every q-tile */
    int64_t kept_total = 0, kept_cap = 0;
    int fail = 0;
    int64_t g = 0; /* global q-tile */

    for (int32_t b = 0; b < batch && !fail; ++b) {
        const int64_t off = cu_seqlens[b];
        const int64_t n = cu_seqlens[b + 1] - off;
        const int64_t nkt = (n + tile - 1) / tile;
        for (int64_t qt = 0; qt * tile < n && !fail; ++qt, ++g) {
            const int32_t *list = ktile_idx + qtile_ptr[g];
            const int64_t len = qtile_ptr[g + 1] - qtile_ptr[g];
            if (len < 0) {
                fail = 1;
                break;
            }
            for (int64_t p = 0; p < len; ++p)
                if (list[p] < 0 || list[p] > qt || (p > 0 && list[p] <= list[p - 1]))
                    fail = 1;
            if (fail)
                break;
            const int64_t r0 = qt * tile;
            const int64_t r1 = (r0 + tile < n) ? r0 + tile : n;
            /* kept k-tiles of the q-tile by brute force over the element mask,
             * appended in increasing order */
            const int64_t first = kept_total;
            for (int64_t kt = 0; kt < nkt && !fail; ++kt) {
                const int64_t c0 = kt * tile;
                const int64_t c1 = (c0 + tile < n) ? c0 + tile : n;
                int any = 0;
                for (int64_t i = r0; i < r1 && !any; ++i)
                    for (int64_t j = c0; j < c1 && !any; ++j)
                        any = oracle_bs_mask(i, j, tile, list, len);
                if (!any)
                    continue;
                if (kept_total == kept_cap) {
                    kept_cap = kept_cap ? 2 * kept_cap : 1024;
                    int32_t *nl = (int32_t *)realloc(kept_list, sizeof(int32_t) * (size_t)kept_cap);
                    if (!nl) {
                        fail = 1;
                        break;
                    }
                    kept_list = nl;
                }
                kept_list[kept_total++] = (int32_t)kt;
            }
            if (fail)
                break;
            /* balanced chunks of at most `bound` tiles, in order */
            const int64_t m = kept_total - first;
            int64_t ns = (m + bound - 1) / bound;
            if (ns < 1)
                ns = 1;
            for (int64_t c = 0; c < ns; ++c) {
                const int64_t a = c * m / ns, z = (c + 1) * m / ns;
                item_t it = {{(int32_t)off, (int32_t)n, (int32_t)r0, (int32_t)r1,
                              (int32_t)(first + a), (int32_t)(z - a), 0, 0, 2,
                              ns > 1 ? (int32_t)(partial_rows + c * (r1 - r0)) : -1,
                              (int32_t)(z - a), 0}};
                fail |= push_item(ns > 1 ? &split_items : &items, &it);
            }
            if (ns > 1) {
                item_t mg = {{(int32_t)off, (int32_t)r0, (int32_t)r1, (int32_t)ns,
                              (int32_t)partial_rows, 0, 0, 0, 0, 0, 0, 0}};
                fail |= push_item(&merges, &mg);
                partial_rows += ns * (r1 - r0);
                merged_rows += r1 - r0;
            }
        }
    }
    int64_t words = -1;
    if (!fail) {
        stable_sort_by_cost(&split_items);
        stable_sort_by_cost(&items);
        const int64_t n_main = split_items.n + items.n;
        words = HDR_WORDS + n_main * ITEM_WORDS + merges.n * MERGE_WORDS + kept_total;
        if (out && cap >= words) {
            const int64_t total = cu_seqlens[batch];
            int32_t *w = out;
            w[0] = SCHED_MAGIC;
            w[1] = SCHED_VERSION;
            w[2] = 2; /* block-sparse */
            w[3] = tile;
            w[4] = batch;
            w[5] = 0;
            w[6] = (int32_t)kept_total; /* length of the appended lists */
            w[7] = 0;
            w[8] = max_tiles;
            w[9] = (int32_t)(uint32_t)((uint64_t)total & 0xffffffffu);
            w[10] = (int32_t)(uint32_t)((uint64_t)total >> 32);
            w[11] = (int32_t)n_main;
            w[12] = (int32_t)merges.n;
            w[13] = (int32_t)partial_rows;
            w[14] = (int32_t)kept_total;
            w[15] = (int32_t)merged_rows;
            w += HDR_WORDS;
            for (int64_t a = 0; a < split_items.n; ++a, w += ITEM_WORDS)
                memcpy(w, split_items.v[a].w, sizeof(int32_t) * ITEM_WORDS);
            for (int64_t a = 0; a < items.n; ++a, w += ITEM_WORDS)
                memcpy(w, items.v[a].w, sizeof(int32_t) * ITEM_WORDS);
            for (int64_t a = 0; a < merges.n; ++a, w += MERGE_WORDS)
                memcpy(w, merges.v[a].w, sizeof(int32_t) * MERGE_WORDS);
            if (kept_total > 0)
                memcpy(w, kept_list, sizeof(int32_t) * (size_t)kept_total);
        }
    }
    free(split_items.v);
    free(items.v);
    free(merges.v);
    free(kept_list);
    return words;
}

/* ---- Region-contribution probe (Sec. 2.2; sections of Appendix A.3) ----
 *
 * The probing variable theta multiplies the attention probabilities
 * elementwise, A_theta = theta (.) A, and the layer output is O = A_theta V.
 * For an upstream gradient dO = d y / d O the derivative at theta = 1 is
 *   d y / d theta_ij = sum_c dO_ic * A_ij * V_jc = A_ij <dO_i, V_j>,
 * and Grad(M-hat, l) is its mean over the pairs of the section M-hat.
 */

static int region_of(int64_t i, int64_t j, int64_t n, int64_t sink,
                     int64_t window, int64_t last)
{
    if (oracle_in_streaming(i, j, sink, window))
        return 0;
    if (oracle_in_middle(i, j, n, sink, window, last))
        return 1;
    if (oracle_in_last(i, j, n, sink, window, last))
        return 2;
    return -1; /* above the diagonal: in no section */
}

int oracle_region_grad(const uint16_t *q, const uint16_t *k, const uint16_t *v,
                       const uint16_t *dout, const double *lse,
                       const int32_t *cu_seqlens, int32_t batch, int32_t hq,
                       int32_t hkv, int32_t d, int64_t sink, int64_t window,
                       int64_t last, double scale, double *sums,
                       double *abs_sums)
{
    if (batch < 0 || hq < 1 || hkv < 1 || hq % hkv != 0 || d < 1 || cu_seqlens[0] != 0)
        return -1;
    for (int32_t b = 0; b < batch; ++b)
        if (cu_seqlens[b + 1] < cu_seqlens[b])
            return -1;
    const int64_t total = cu_seqlens[batch];
    const int32_t group = hq / hkv;
    int bad = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(| : bad)
    for (int32_t h = 0; h < hq; ++h) {
        const int32_t g = h / group;
        double acc[3] = {0, 0, 0}, acc_abs[3] = {0, 0, 0};
        double *qi = (double *)malloc(sizeof(double) * (size_t)d);
        double *di = (double *)malloc(sizeof(double) * (size_t)d);
        if (!qi || !di) {
            bad = 1;
            free(qi);
            free(di);
            continue;
        }
        for (int32_t b = 0; b < batch; ++b) {
            const int64_t off = cu_seqlens[b];
            const int64_t n = cu_seqlens[b + 1] - off;
            for (int64_t i = 0; i < n; ++i) {
                const int64_t ti = off + i;
                for (int32_t c = 0; c < d; ++c) {
                    qi[c] = widen_bf16(q[(ti * hq + h) * d + c]);
                    di[c] = widen_bf16(dout[(ti * hq + h) * d + c]);
                }
                const double lse_i = lse[(int64_t)h * total + ti];
                for (int64_t j = 0; j <= i; ++j) {
                    const int r = region_of(i, j, n, sink, window, last);
                    if (r < 0)
                        continue;
                    const int64_t tj = off + j;
                    double z = 0.0, gv = 0.0;
                    for (int32_t c = 0; c < d; ++c) {
                        z += qi[c] * widen_bf16(k[(tj * hkv + g) * d + c]);
                        gv += di[c] * widen_bf16(v[(tj * hkv + g) * d + c]);
                    }
                    const double a = exp(scale * z - lse_i);
                    acc[r] += a * gv;
                    acc_abs[r] += fabs(a * gv);
                }
            }
        }
        for (int r = 0; r < 3; ++r) {
            sums[h * 3 + r] = acc[r];
            if (abs_sums)
                abs_sums[h * 3 + r] = acc_abs[r];
        }
        free(qi);
        free(di);
    }
    return bad ? -1 : 0;
}

int oracle_region_counts(const int32_t *cu_seqlens, int32_t batch, int64_t sink,
                         int64_t window, int64_t last, int64_t *counts)
{
    if (batch < 0 || cu_seqlens[0] != 0)
        return -1;
    counts[0] = counts[1] = counts[2] = 0;
    for (int32_t b = 0; b < batch; ++b) {
        const int64_t n = cu_seqlens[b + 1] - cu_seqlens[b];
        if (n < 0)
            return -1;
        for (int64_t i = 0; i < n; ++i)
            for (int64_t j = 0; j <= i; ++j) {
                const int r = region_of(i, j, n, sink, window, last);
                if (r >= 0)
                    ++counts[r];
            }
    }
    return 0;
}

int oracle_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
