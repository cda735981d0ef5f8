/*
 * oracle.h -- plain, slow, fp64 CPU reference for Triangle attention and
 * dense causal attention (arXiv 2507.21526).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may include, link
 * or call this code: it exists so that tests, the smoke check and the CPU
 * baseline leg of the benchmark can check the HIP library against the
 * paper's definitions.  It shares no source with the library.
 *
 * Conventions (the readings are listed with their reasons in the design
 * notes of the repository):
 *   - rows i and keys j are 0-indexed inside one sequence of length n;
 *   - sink   = keys j < S                         (Appendix A.3, M-stream)
 *   - window = keys with 0 <= i - j < W            (Appendix A.3, M-stream)
 *   - Last   = rows i >= n - min(L, n)             (Appendix A.3, M-last)
 *   - Triangle mask = M-stream OR M-last = causal minus M-middle (Sec. 2.4)
 *   - masked logits are removed exactly (Sec. 2.1, the -c(1-M) term with
 *     c -> infinity), never weighted by a finite exp(-c).
 *   - GQA: query head h reads kv head floor(h / G), G = Hq / Hkv.
 * Inputs are bf16 bit patterns (uint16); every value is widened exactly to
 * double before use.
 */
#ifndef TRIANGLE_ORACLE_H
#define TRIANGLE_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { ORACLE_TRIANGLE = 0, ORACLE_CAUSAL = 1 };

/* Region predicates of Appendix A.3 (one sequence of length n). */
int oracle_in_streaming(int64_t i, int64_t j, int64_t sink, int64_t window);
int oracle_in_last(int64_t i, int64_t j, int64_t n, int64_t sink,
                   int64_t window, int64_t last);
int oracle_in_middle(int64_t i, int64_t j, int64_t n, int64_t sink,
                     int64_t window, int64_t last);
/* Mask of the pass: Triangle = streaming OR last; causal = (j <= i). */
int oracle_mask(int kind, int64_t i, int64_t j, int64_t n, int64_t sink,
                int64_t window, int64_t last);

/* Materialise mask row i of a length-n sequence into row[0..n). */
void oracle_mask_row(int kind, int64_t n, int64_t sink, int64_t window,
                     int64_t last, int64_t i, uint8_t *row);

/* Number of kept (i, j) pairs of one sequence (one head). */
int64_t oracle_mask_nnz(int kind, int64_t n, int64_t sink, int64_t window,
                        int64_t last);

/*
 * Attention rows by the plain definition (Sec. 2.1, masked softmax):
 *   z_j = scale * <q_i, k_j> for kept j;  p = softmax(z);  out = sum_j p_j v_j;
 *   lse = log(sum_j exp(z_j))  (natural log).
 * q: [total, hq, d], k and v: [total, hkv, d], bf16 bits, packed by
 * cu_seqlens[batch + 1].  Row r of the request is (token row_tok[r], query
 * head row_head[r]); out[r * d .. r * d + d) and lse[r] receive its result.
 * Returns 0, or -1 on an invalid request (token out of range, bad heads).
 * Parallel over requested rows with OpenMP.
 */
int oracle_attn_rows(const uint16_t *q, const uint16_t *k, const uint16_t *v,
                     const int32_t *cu_seqlens, int32_t batch, int32_t hq,
                     int32_t hkv, int32_t d, int kind, int64_t sink,
                     int64_t window, int64_t last, double scale,
                     const int64_t *row_tok, const int32_t *row_head,
                     int64_t nrows, double *out, double *lse);

/*
 * oracle_attn_rows plus, per output element, the probability-weighted mean
 * of |v| over the row's kept keys: absw[r * d + c] = sum_j p_j |v_jc|.  It
 * bounds the error that rounding the probabilities to a narrower format
 * can cause in a weighted sum of V: if each p_j carries a relative error of
 * at most u, the output element moves by at most u * absw (numerator only;
 * the normaliser is kept exact).
 */
int oracle_attn_rows_absw(const uint16_t *q, const uint16_t *k, const uint16_t *v,
                          const int32_t *cu_seqlens, int32_t batch, int32_t hq,
                          int32_t hkv, int32_t d, int kind, int64_t sink,
                          int64_t window, int64_t last, double scale,
                          const int64_t *row_tok, const int32_t *row_head,
                          int64_t nrows, double *out, double *lse, double *absw);

/*
 * Tile schedule by brute force: a (q-tile, k-tile) pair is kept iff some
 * (i, j) inside it is kept by oracle_mask.  Emitted in the documented packed
 * int32 format (header, main items, merge items).  Writes at most cap words
 * into out (out may be NULL for a size query) and returns the number of
 * words the schedule needs, or -1 on invalid parameters.
 */
int64_t oracle_schedule(int kind, const int32_t *cu_seqlens, int32_t batch,
                        int32_t sink, int32_t window, int32_t last,
                        int32_t tile, int32_t splits, int32_t *out,
                        int64_t cap);

/*
 * Block-sparse causal attention (Sec. 2.4 / Sec. 3.1: the dense layers handed
 * to a dynamic sparse method, whose estimator lists the kept k-tiles of each
 * q-tile).  Lists are CSR over the q-tiles of all sequences in order
 * (q-tile t of sequence b has global index sum_{b' < b} ceil(n_b' / tile) + t):
 * the k-tiles of global q-tile g are ktile_idx[qtile_ptr[g] .. qtile_ptr[g+1]).
 * Row i keeps key j iff j <= i and floor(j / tile) is listed for q-tile
 * floor(i / tile).  A row with no kept key has output 0 and lse -inf.
 */
int oracle_bs_mask(int64_t i, int64_t j, int64_t tile, const int32_t *list,
                   int64_t len);
int oracle_attn_rows_bs(const uint16_t *q, const uint16_t *k, const uint16_t *v,
                        const int32_t *cu_seqlens, int32_t batch, int32_t hq,
                        int32_t hkv, int32_t d, int32_t tile,
                        const int32_t *qtile_ptr, const int32_t *ktile_idx,
                        double scale, const int64_t *row_tok,
                        const int32_t *row_head, int64_t nrows, double *out,
                        double *lse);
/*
 * Region-contribution probe (Sec. 2.2, Grad(M-hat, l)).  The probing
 * variable theta scales the attention probabilities elementwise; for an
 * upstream gradient dO of the attention output the derivative at theta = 1
 * is A_ij <dO_i, V_j>, with A_ij = exp(scale <q_i, k_j> - lse_i).  For every
 * query head h and section r of Appendix A.3 (0 streaming, 1 middle, 2 last;
 * together the causal mask):
 *   sums[h * 3 + r]     = sum over (i, j) in section r of A_ij <dO_i, V_j>
 *   abs_sums[h * 3 + r] = sum of |A_ij <dO_i, V_j>| (may be NULL).
 * q, dout: [total, hq, d]; k, v: [total, hkv, d] (bf16 bits); lse: [hq,
 * total] natural log, the row normaliser to use (the causal one for a dense
 * layer).  Grad = sums / the section's pair count (oracle_region_counts).
 * OpenMP over heads.  Returns 0, or -1 on invalid arguments.
 */
int oracle_region_grad(const uint16_t *q, const uint16_t *k, const uint16_t *v,
                       const uint16_t *dout, const double *lse,
                       const int32_t *cu_seqlens, int32_t batch, int32_t hq,
                       int32_t hkv, int32_t d, int64_t sink, int64_t window,
                       int64_t last, double scale, double *sums,
                       double *abs_sums);

/* Pairs (i, j) per head in each section (streaming, middle, last), summed
 * over the sequences, by brute force.  Returns 0, or -1 on invalid input. */
int oracle_region_counts(const int32_t *cu_seqlens, int32_t batch, int64_t sink,
                         int64_t window, int64_t last, int64_t *counts);

/*
 * Block-sparse schedule in the packed format: the kept k-tiles of each
 * q-tile found by brute force over oracle_bs_mask, cut in order into
 * ns = max(1, ceil(m / bound)) balanced chunks (bound = max_tiles, or when
 * it is 0: max(16, ceil(2 * listed tiles / q-tiles))), one
 * list item (mode 2: ka0 = offset into the appended lists, ka1 = length)
 * per chunk; q-tiles with several items get split items and a merge item;
 * split items first, then the rest, each stable by decreasing tiles; the
 * kept k-tiles of every q-tile appended in q-tile order (header word 6 holds
 * their count).  Returns the number of words, or -1 on invalid lists.
 */
int64_t oracle_bs_schedule(const int32_t *cu_seqlens, int32_t batch,
                           int32_t tile, const int32_t *qtile_ptr,
                           const int32_t *ktile_idx, int32_t max_tiles,
                           int32_t *out, int64_t cap);

int oracle_num_threads(void);

#ifdef __cplusplus
}
#endif
#endif
