/*
 * triattn.h -- C interface of the MI355X (gfx950) Triangle attention library.
 *
 * Triangle attention is the static sparse prefill attention of TriangleMix
 * (arXiv 2507.21526, Sec. 2.4): every query attends to the Streaming section
 * (the first `sink` keys plus a causal window of `window` keys) and the last
 * `last` queries of each sequence attend causally to every key (Last Q-K
 * section, Appendix A.3); the Middle Q-K section is skipped.  Dense causal
 * attention (Sec. 2.1 with the causal mask) is the path of the layers that
 * stay dense.  The forward passes follow the split structure of Appendix A.1
 * (Algorithm "Fused Triangle Attention"): streaming q-tiles over their sink
 * and window k-tiles, the Last rows split over the key range, and an
 * LSE-weighted merge of the split partials.  The library also runs
 * block-sparse causal attention over caller-listed k-tiles (the dense layers
 * handed to a dynamic sparse method, Sec. 2.4 and 3.1) and the
 * region-contribution probe that chooses the Triangle layers (Sec. 2.2 and
 * 3).
 *
 * Conventions
 *   - Rows i and keys j are 0-indexed within a sequence of length n.  A
 *     Triangle row keeps key j iff j <= i and (j < sink or i - j < window or
 *     i >= n - min(last, n)).  Masked logits are excluded exactly.
 *   - Tensors are packed "THD": q and o are [total_tokens, hq, head_dim],
 *     k and v are [total_tokens, hkv, head_dim], contiguous, bf16 (o may be
 *     fp32), 16-byte aligned device pointers.  Sequences are packed by
 *     cu_seqlens[batch + 1] (cu_seqlens[0] = 0, non-decreasing).
 *   - GQA: query head h reads kv head h / (hq / hkv).
 *   - lse, when not NULL, is [hq, total_tokens] fp32: natural-log
 *     log-sum-exp of the kept scaled logits of each row.
 *   - Supported: head_dim in {64, 128}, tile in {64, 128}, hq % hkv == 0,
 *     hq / hkv <= 8.  Others return TA_ERR_UNSUPPORTED.
 *
 * Ownership and synchronisation
 *   The caller owns every buffer (inputs, outputs, the device copy of the
 *   schedule, the workspace).  The forward functions allocate nothing, keep
 *   no pointer after they return, never synchronise, and enqueue their
 *   kernels on the caller's stream (a hipStream_t passed as void*; NULL is
 *   the default stream).  Execution faults surface at the caller's next
 *   synchronisation.
 *
 * Errors
 *   Every argument is checked before any launch.  On error a function
 *   returns a nonzero ta_status, launches nothing, leaves every output
 *   untouched and records a message that ta_last_error() returns (per
 *   thread).  No C++ exception crosses this interface.  The kernels also
 *   check the device schedule against the launch arguments: a header that
 *   does not match makes every workgroup fill its share of O (and LSE) with
 *   NaN, so that every element is NaN; an item whose words are out of range
 *   or whose mode the launch does not serve is not computed, and its
 *   workgroups fill the rows it names (clamped into the buffers, one q-tile
 *   at most) with NaN, so that the failure is visible in the output.  No
 *   access leaves the caller's buffers either way.
 */
#ifndef TRIATTN_H
#define TRIATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define TA_ABI_VERSION 3
#define TA_SCHEDULE_MAGIC 0x54524941
#define TA_SCHEDULE_VERSION 2

typedef enum {
    TA_OK = 0,
    TA_ERR_INVALID_ARG = 1,      /* NULL pointer, negative size, bad enum */
    TA_ERR_UNSUPPORTED = 2,      /* valid but not implemented (head_dim...) */
    TA_ERR_BUFFER_TOO_SMALL = 3, /* schedule output buffer too small */
    TA_ERR_WORKSPACE = 4,        /* workspace missing or too small */
    TA_ERR_SCHEDULE_MISMATCH = 5,/* info does not fit the call */
    TA_ERR_HIP = 6               /* a HIP launch call failed */
} ta_status;

typedef enum {
    TA_KIND_TRIANGLE = 0,   /* Triangle attention (ta_build_schedule) */
    TA_KIND_CAUSAL = 1,     /* dense causal attention (ta_build_schedule) */
    TA_KIND_BLOCKSPARSE = 2 /* caller-listed k-tiles (ta_build_blocksparse_schedule) */
} ta_kind;
typedef enum { TA_OUT_BF16 = 0, TA_OUT_F32 = 1 } ta_out_dtype;

/* Summary of a built schedule (mirrors the header words of the packed form). */
typedef struct ta_schedule_info {
    int32_t version;          /* TA_SCHEDULE_VERSION */
    int32_t kind;             /* ta_kind */
    int32_t tile;             /* T: q-tile rows = k-tile keys */
    int32_t batch;
    int32_t sink, window, last;
    int32_t splits_requested; /* 0 = automatic split rule */
    int64_t total_tokens;
    int64_t words;            /* int32 words of the packed schedule */
    int32_t n_items;          /* main-pass work items (split items first) */
    int32_t n_last_items;     /* of which split items (Last rows or split
                                 block-sparse q-tiles) */
    int32_t n_merge_items;    /* split q-tiles (one merge each) */
    int32_t n_last_rows;      /* rows covered by merge items */
    int32_t n_partial_rows;   /* rows of split partials in the workspace */
    int32_t max_splits;       /* largest split count of a q-tile */
    int64_t kept_tiles_per_qhead; /* kept (q-tile, k-tile) pairs per head */
    int32_t max_item_tiles;   /* most k-tiles of one work item (sizes the
                                 launch of the attention pass) */
    int32_t reserved;         /* 0 */
} ta_schedule_info;

/* Library interface version (TA_ABI_VERSION). */
int32_t ta_abi_version(void);

/* Message of the last non-OK status returned on this thread ("" if none). */
const char *ta_last_error(void);

/*
 * Build the tile schedule of a pass on the host (Appendix A.1: which k-tiles
 * each q-tile visits; Appendix A.3: the sections they cover).
 *   kind        TA_KIND_TRIANGLE or TA_KIND_CAUSAL.
 *   cu_seqlens  host array of batch + 1 int32 (cu_seqlens[0] = 0,
 *               non-decreasing, cu_seqlens[batch] = total tokens).
 *   sink >= 0, window >= 1, last >= 0 (Triangle; stored but unused for
 *               causal).  last = 0 gives the Streaming pattern.
 *   tile        64 or 128.
 *   splits      0 = automatic: a Last q-tile with nk kept k-tiles gets
 *               ceil(nk / t) splits (at most nk), t = max(ceil(sink/tile) +
 *               ceil(window/tile) + 1, ceil(2048/tile)); > 0 = that many
 *               (at most nk).
 *   out         host buffer of out_words int32, or NULL to query the size
 *               (info is filled either way).
 * Returns TA_OK, TA_ERR_INVALID_ARG, TA_ERR_UNSUPPORTED or
 * TA_ERR_BUFFER_TOO_SMALL (info->words then holds the size needed).
 * The caller copies `out` to device memory for the forward call.
 */
ta_status ta_build_schedule(int32_t kind, const int32_t *cu_seqlens,
                            int32_t batch, int32_t sink, int32_t window,
                            int32_t last, int32_t tile, int32_t splits,
                            int32_t *out, int64_t out_words,
                            ta_schedule_info *info);

/*
 * Build the schedule of block-sparse causal attention on the host: the same
 * tile passes driven by a caller-supplied list of kept k-tiles per q-tile.
 * This is the attention of the layers TriangleMix keeps dense when they are
 * handed to a dynamic sparse method instead (Sec. 2.4; the "Ours + X"
 * combinations of Sec. 3.1), whose index estimator produces such lists.
 *   Row i (0-indexed in its sequence, q-tile i / tile) keeps key j iff
 *   j <= i and k-tile j / tile is listed for that q-tile.  A row that keeps
 *   no key gets a zero output row and lse = -inf.
 *   cu_seqlens  as for ta_build_schedule.
 *   tile        64 or 128.
 *   qtile_ptr   host array of Q + 1 int32, Q = sum over sequences of
 *               ceil(n_b / tile) (q-tiles in sequence order): the k-tiles of
 *               global q-tile t are ktile_idx[qtile_ptr[t] .. qtile_ptr[t+1]).
 *               qtile_ptr[0] = 0, non-decreasing.
 *   ktile_idx   host array of sequence-relative k-tile indices, strictly
 *               increasing per q-tile, each in [0, q-tile index] (tiles
 *               above the diagonal hold no key j <= i and are rejected).
 *               May be NULL when every list is empty.
 *   max_tiles_per_item  work bound per item; 0 = automatic: max(16,
 *               ceil(2 * listed tiles / q-tiles)), so only lists longer
 *               than twice the mean are cut.  The list of a q-tile with m
 *               tiles is cut, in order, into ns = max(1, ceil(m / bound))
 *               balanced chunks (chunk c holds list entries
 *               [c m / ns, (c + 1) m / ns)); each chunk is one work item.  A
 *               q-tile with one item writes its rows directly; one with
 *               several gets split items (normalised fp32 partials in the
 *               workspace) and a merge item, as the Last rows of Triangle
 *               attention.  Items are ordered split items first, each group
 *               by decreasing tile count (stable); merge items in q-tile
 *               order.  The lists themselves are appended to the schedule.
 *   out, out_words, info  as for ta_build_schedule; info->kind is
 *               TA_KIND_BLOCKSPARSE, sink = last = 0, window = the number of
 *               listed k-tiles (the length of the appended lists) and
 *               splits_requested = max_tiles_per_item.
 */
ta_status ta_build_blocksparse_schedule(const int32_t *cu_seqlens, int32_t batch,
                                        int32_t tile, const int32_t *qtile_ptr,
                                        const int32_t *ktile_idx,
                                        int32_t max_tiles_per_item, int32_t *out,
                                        int64_t out_words, ta_schedule_info *info);

/* Bytes of workspace triangle_attn_fwd (or blocksparse_attn_fwd) needs for
 * the split partials (fp32 partial outputs and their LSE); 0 when there are
 * none. */
size_t ta_workspace_bytes(const ta_schedule_info *info, int32_t hq,
                          int32_t head_dim);

/*
 * Triangle attention forward (Sec. 2.4; Appendix A.1 and A.3).
 *   q, k, v      bf16 device tensors in THD layout (see above).
 *   o            [total_tokens, hq, head_dim], bf16 or fp32 per o_dtype.
 *   lse          [hq, total_tokens] fp32 or NULL.
 *   sched_dev    device copy of the words built by ta_build_schedule with
 *                kind TA_KIND_TRIANGLE; info is the matching summary.
 *   softmax_scale  multiplies q.k (1/sqrt(head_dim) in the paper).
 *   workspace    device buffer of at least ta_workspace_bytes() bytes
 *                (may be NULL when that is 0); its contents on entry do
 *                not matter.
 * Every output row (and lse entry) is written exactly once.
 */
ta_status triangle_attn_fwd(const void *q, const void *k, const void *v,
                            void *o, int32_t o_dtype, float *lse,
                            const int32_t *sched_dev,
                            const ta_schedule_info *info, int64_t total_tokens,
                            int32_t hq, int32_t hkv, int32_t head_dim,
                            float softmax_scale, void *workspace,
                            size_t workspace_bytes, void *stream);

/*
 * Triangle attention forward without a caller workspace, for callers that
 * cannot allocate device memory (code under HIP graph capture, serving loops
 * or harnesses that forbid hipMalloc).  Same arguments and results as
 * triangle_attn_fwd minus the workspace: the Last-row split partials go to a
 * library-owned device array of TA_NOALLOC_SCRATCH_BYTES bytes per GPU,
 * reserved when the library's code is loaded on that GPU and held until the
 * process ends.  The first call on a GPU looks up the array's address (a HIP
 * call, no allocation); no call allocates or frees memory.
 *   Limit: ta_workspace_bytes(info, hq, head_dim) must not exceed
 *   TA_NOALLOC_SCRATCH_BYTES (otherwise TA_ERR_WORKSPACE, nothing launched);
 *   e.g. 128 Last rows x 32 heads x 57 splits at head_dim 128 take 120.5 MB.
 *   Pass a smaller explicit split count to ta_build_schedule to fit.
 *   Sharing: every call on one GPU uses the same array.  The partials are
 *   written before they are read within a call, so nothing needs clearing,
 *   but calls that overlap on one GPU (concurrent streams, threads) race.
 */
#define TA_NOALLOC_SCRATCH_BYTES (128u << 20)
ta_status triangle_attn_fwd_noalloc(const void *q, const void *k, const void *v,
                                    void *o, int32_t o_dtype, float *lse,
                                    const int32_t *sched_dev,
                                    const ta_schedule_info *info,
                                    int64_t total_tokens, int32_t hq, int32_t hkv,
                                    int32_t head_dim, float softmax_scale,
                                    void *stream);

/*
 * The two passes of triangle_attn_fwd, callable on their own (same stream
 * order: tiles, then merge); triangle_attn_fwd is exactly these two calls.
 *
 * triangle_attn_tiles: the attention pass over every schedule item (Appendix
 *   A.1: streaming q-tiles over their sink and window k-tiles; Last q-tiles
 *   split over the key range).  Streaming rows go to o (and lse); Last rows
 *   go to the workspace as normalised fp32 partial outputs with their LSE.
 *   Arguments as triangle_attn_fwd.
 * triangle_attn_merge: LSE-weighted merge of the split partials of every
 *   Last row into o (and lse) (Appendix A.1, merge of the last-row buffers):
 *   O = sum_c w_c O_c / sum_c w_c with w_c = exp(LSE_c - max_c LSE_c), and
 *   LSE = max_c LSE_c + log(sum_c w_c).  Reads the workspace written by
 *   triangle_attn_tiles with the same schedule, hq and head_dim.
 */
ta_status triangle_attn_tiles(const void *q, const void *k, const void *v,
                              void *o, int32_t o_dtype, float *lse,
                              const int32_t *sched_dev,
                              const ta_schedule_info *info,
                              int64_t total_tokens, int32_t hq, int32_t hkv,
                              int32_t head_dim, float softmax_scale,
                              void *workspace, size_t workspace_bytes,
                              void *stream);
ta_status triangle_attn_merge(void *o, int32_t o_dtype, float *lse,
                              const int32_t *sched_dev,
                              const ta_schedule_info *info,
                              int64_t total_tokens, int32_t hq,
                              int32_t head_dim, const void *workspace,
                              size_t workspace_bytes, void *stream);

/*
 * Dense causal attention forward (Sec. 2.1 with the causal mask), the
 * attention of the layers TriangleMix keeps dense.  Same arguments as
 * triangle_attn_fwd; the schedule must be built with TA_KIND_CAUSAL.  Needs
 * no workspace.
 */
ta_status causal_attn_fwd(const void *q, const void *k, const void *v,
                          void *o, int32_t o_dtype, float *lse,
                          const int32_t *sched_dev,
                          const ta_schedule_info *info, int64_t total_tokens,
                          int32_t hq, int32_t hkv, int32_t head_dim,
                          float softmax_scale, void *stream);

/*
 * Block-sparse causal attention forward over a TA_KIND_BLOCKSPARSE schedule
 * (Sec. 2.4 and 3.1, "Ours + X": the dense layers replaced by a dynamic
 * sparse method): the tile pass over every item, then the LSE-weighted merge
 * of the split q-tiles.  Same arguments and workspace rule as
 * triangle_attn_fwd.
 */
ta_status blocksparse_attn_fwd(const void *q, const void *k, const void *v,
                               void *o, int32_t o_dtype, float *lse,
                               const int32_t *sched_dev,
                               const ta_schedule_info *info, int64_t total_tokens,
                               int32_t hq, int32_t hkv, int32_t head_dim,
                               float softmax_scale, void *workspace,
                               size_t workspace_bytes, void *stream);

/*
 * Region-contribution probe (Sec. 2.2, Grad(M-hat, l); the sections of
 * Appendix A.3).  A probing variable theta scales the attention
 * probabilities elementwise (A_theta = theta (.) A, O = A_theta V); for an
 * upstream gradient dO = dy/dO of the attention output, the derivative at
 * theta = 1 is  dy / dtheta_ij = A_ij <dO_i, V_j>.  This call sums it, for
 * every query head h and section r (0 streaming, 1 middle, 2 last; together
 * the causal pairs j <= i of every sequence), into
 *   region_sums[h * 3 + r]   (fp64 device array of hq * 3 values).
 * A_ij = exp(softmax_scale <q_i, k_j> - lse_i) is recomputed from q, k and
 * the given row normaliser.
 *   q, dout      [total_tokens, hq, head_dim] bf16; k, v [total_tokens, hkv,
 *                head_dim] bf16; all 16-byte aligned.
 *   lse          [hq, total_tokens] fp32, natural log: the causal softmax
 *                normaliser of each row (causal_attn_fwd writes it).
 *   sched_dev, info  a TA_KIND_CAUSAL schedule of the same cu_seqlens (its
 *                work items are the tiles the probe visits).
 *   sink, window, last  the sections (sink = keys j < sink, window = keys
 *                with i - j < window, last = rows i >= n - min(last, n) of
 *                each sequence); all >= 0.  The paper probes with 64, 128,
 *                128 on ~2K-token prompts.
 *   workspace    device buffer of at least ta_probe_workspace_bytes(info,
 *                hq) bytes (512 * tile / 32 * hq * 3 doubles; 0 for a
 *                schedule without items), 8-byte aligned (NULL when that is
 *                0); its contents on entry do not matter.
 * Grad(M-hat_r, l) = sum_h region_sums[h * 3 + r] / (hq * count_r) with the
 * pair counts of ta_region_counts (ta_region_grad_mean).  The work is cut
 * into equal shares of kept 64-key steps (plus a charge per q-tile change),
 * one per workgroup, so the pass does not wait on the longest q-tile.  The
 * result is deterministic (fixed shares and reduction order for a given
 * shape).  Device schedule words that do not
 * match info give NaN sums.  Errors as triangle_attn_fwd.
 */
size_t ta_probe_workspace_bytes(const ta_schedule_info *info, int32_t hq);
ta_status region_grad_probe(const void *q, const void *k, const void *v,
                            const void *dout, const float *lse,
                            const int32_t *sched_dev,
                            const ta_schedule_info *info, int64_t total_tokens,
                            int32_t hq, int32_t hkv, int32_t head_dim,
                            float softmax_scale, int32_t sink, int32_t window,
                            int32_t last, double *region_sums, void *workspace,
                            size_t workspace_bytes, void *stream);

/*
 * Host helpers of the probe (Appendix A.3 sections; Sec. 3 layer choice).
 * ta_region_counts: pairs (i, j) per head in each section (streaming,
 *   middle, last), summed over the sequences of cu_seqlens[batch + 1]
 *   (host array); counts is a host array of 3.
 * ta_region_grad_mean: grad[r] = sum_h region_sums[h * 3 + r] / (hq *
 *   counts[r]) (0 for an empty section); host arrays.
 * ta_select_triangle_layers: the n_triangle layers whose middle-section
 *   value has the smallest magnitude (ties: lower layer first), written to
 *   layers[0 .. n_triangle) in increasing order.  Values must be finite.
 */
ta_status ta_region_counts(const int32_t *cu_seqlens, int32_t batch,
                           int32_t sink, int32_t window, int32_t last,
                           int64_t *counts);
ta_status ta_region_grad_mean(const double *region_sums, int32_t hq,
                              const int64_t *counts, double *grad);
ta_status ta_select_triangle_layers(const double *grad_middle,
                                    int32_t n_layers, int32_t n_triangle,
                                    int32_t *layers);

#ifdef __cplusplus
}
#endif
#endif /* TRIATTN_H */
