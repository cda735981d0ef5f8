// HIP forward passes of libtriattn.so for gfx950 (MI355X).
//
// One tile kernel serves the three attention passes of the schedule:
//   * streaming q-tiles of Triangle attention (sink and window k-tiles,
//     Appendix A.1 upper part; streaming mask of Appendix A.3),
//   * Last-row split items (one contiguous chunk of k-tiles of a Last q-tile,
//     Appendix A.1 lower part), writing normalised fp32 partials and LSE,
//   * q-tiles of dense causal attention (Sec. 2.1, causal mask).
// A second kernel merges the split partials of the Last rows with LSE
// weights (Appendix A.1, merge of the last-row buffers).
//
// Tile core (flash-style online softmax, Sec. 2.1 evaluated blockwise):
//   A workgroup owns one work item, one kv head g and R query rows of each of
//   the G query heads of g, so every K/V tile staged in LDS is shared by the
//   whole GQA group.  Each wave owns 32 query rows of one head.  Keys advance
//   in steps of 64.  The wave computes S^T = K Q^T with bf16 MFMA 32x32x16
//   (keys on the MFMA rows, queries on the columns), so a lane holds 32
//   scores of a single query: the softmax max/sum are in-lane plus one swap
//   between the two lane halves.  The K rows fed to the MFMA are permuted
//   (bits 2 and 3 of the row index swapped) so that the score registers are
//   directly the B operand of O^T += V^T P^T, with V staged transposed in
//   LDS.  Softmax runs in the log2 domain with fp32 state.
//
// Q enters and bf16 O leaves through LDS in whole rows (the MFMA register
// layout would touch 32 rows per load or store instruction); each workgroup
// trims its key runs to the steps its own rows can reach; a block-sparse
// list item reads its step keys from the list once, into an LDS table.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstdlib>
#include <mutex>
#include <type_traits>

#include "triattn_device.h"
#include "triattn_internal.h"

// Library-owned device memory of triangle_attn_fwd_noalloc: the Last-row
// split partials (fp32 partial outputs, then their LSE, laid out as in a
// caller's workspace).  Each GPU the library runs on holds its own copy
// until the process ends.  In host code this name is only a handle for
// hipGetSymbolAddress: kernels receive the device address obtained from it.
static __device__ __align__(256) unsigned char scratch[TA_NOALLOC_SCRATCH_BYTES];

namespace triattn {
namespace {

typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

constexpr int kStep = 64;  // keys per inner step
constexpr int kKeyTable = 2048;  // LDS table of a list item's step keys
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

struct FwdArgs {
    const uint16_t *q;
    const uint16_t *k;
    const uint16_t *v;
    void *o;
    float *lse;
    const int32_t *sched;
    float *part_o;    // [partial rows, hq, d] fp32
    float *part_lse;  // [partial rows, hq] fp32
    int64_t total_tokens;
    int32_t hq, hkv, group;
    int32_t n_items;
    int32_t n_partial_rows;
    int64_t list_base;    // first word of the k-tile lists (after the merges)
    int64_t list_words;   // words in the k-tile lists
    int32_t sink, window;
    int32_t tile;
    int32_t rows_per_wg;  // R
    int32_t subtiles;     // tile / R
    int32_t o_f32;
    float scale_log2;     // softmax scale * log2(e)
    // multi-unit kernel: units = items x subtiles per kv head; workgroup
    // (slot, head) runs units slot, slot + n_slots, ... (at most upw)
    int32_t n_units;
    int32_t n_slots;
    int32_t upw;
    // single-unit kernel: the first n_lead items (a Triangle schedule's Last
    // split items) are interleaved with the others in launch order (0: none)
    int32_t n_lead;
};

struct MergeArgs {
    const int32_t *sched;
    const float *part_o;
    const float *part_lse;
    void *o;
    float *lse;
    int64_t total_tokens;
    int32_t hq;
    int32_t n_items;
    int32_t n_merges;
    int32_t n_partial_rows;
    int32_t n_last_rows;
    int32_t o_f32;
    int32_t kind;  // schedule kind the merge items come from
    int32_t tile;  // rows of a merge item are at most one q-tile
};

// The tests combine with & (no short-circuit), so every header word is
// loaded before any test: the loads go out together instead of one memory
// round trip per test.
__device__ __forceinline__ bool header_ok(const int32_t *s, int64_t total,
                                          int32_t n_items, int32_t kind)
{
    const int64_t t = (int64_t)(uint32_t)s[H_TOTAL_LO] |
                      ((int64_t)s[H_TOTAL_HI] << 32);
    return (s[H_MAGIC] == TA_SCHEDULE_MAGIC) & (s[H_VERSION] == TA_SCHEDULE_VERSION) &
           (s[H_KIND] == kind) & (t == total) & (s[H_ITEMS] == n_items);
}

// A schedule that does not match the launch (wrong header, malformed item)
// leaves the workgroup without rows it can trust: every workgroup that finds
// one fills its slice of O (and of LSE) with NaN instead, the slices of the
// whole grid together covering every element, so that the caller sees the
// failure in the output (Appendix A.1 initialises O before the loops; here
// a rejected schedule leaves it NaN, not stale).  Vector stores only.
__device__ __forceinline__ void poison_outputs(void *o, int o_f32, float *lse,
                                            int64_t total_tokens, int32_t hq, int d,
                                            int64_t block, int64_t n_blocks)
{
    const int64_t n_o = total_tokens * hq * d;
    const int64_t n_l = lse ? total_tokens * hq : 0;
    const int64_t co = (n_o + n_blocks - 1) / n_blocks;
    const int64_t cl = (n_l + n_blocks - 1) / n_blocks;
    const int64_t o0 = block * co, o1 = min(o0 + co, n_o);
    const int64_t l0 = block * cl, l1 = min(l0 + cl, n_l);
    for (int64_t i = o0 + threadIdx.x; i < o1; i += blockDim.x) {
        if (o_f32)
            reinterpret_cast<float *>(o)[i] = __builtin_nanf("");
        else
            reinterpret_cast<uint16_t *>(o)[i] = 0x7fc0;  // bf16 quiet NaN
    }
    for (int64_t i = l0 + threadIdx.x; i < l1; i += blockDim.x)
        lse[i] = __builtin_nanf("");
}

// A rejected item's own rows (every head), as far as its words say where
// they are (clamped into the buffers, one q-tile at most), filled with NaN,
// and its split partial rows when it names some: no other workgroup writes
// these rows (a split item's O rows are the merge's, which then reads the
// NaN partials), so a malformed item is visible in O and LSE, which the
// slice of poison_outputs alone does not ensure (later workgroups may
// overwrite that slice).  Every index stays inside the buffers the host
// checked, whatever the words hold.
__device__ __forceinline__ void poison_item_rows(void *o, int o_f32, float *lse, float *part_o,
                                                 float *part_lse, int64_t total_tokens,
                                                 int32_t hq, int d, int64_t n_partial_rows,
                                                 int tile, int64_t seq_off, int64_t r0,
                                                 int64_t r1, int64_t part_base)
{
    const int64_t lo = min(max(seq_off + r0, (int64_t)0), total_tokens);
    int64_t hi = min(max(seq_off + r1, lo), lo + tile);
    if (hi == lo)
        hi = lo + tile;  // an empty or reversed row range: the tile from lo
    hi = min(hi, total_tokens);
    const int64_t rows = hi - lo;
    for (int64_t i = threadIdx.x; i < rows * hq * d; i += blockDim.x) {
        if (o_f32)
            reinterpret_cast<float *>(o)[lo * hq * d + i] = __builtin_nanf("");
        else
            reinterpret_cast<uint16_t *>(o)[lo * hq * d + i] = 0x7fc0;  // bf16 quiet NaN
    }
    if (lse)
        for (int64_t i = threadIdx.x; i < rows * hq; i += blockDim.x)
            lse[(i / rows) * total_tokens + lo + i % rows] = __builtin_nanf("");
    if (part_o && part_base >= 0 && part_base < n_partial_rows) {
        const int64_t prows = min(rows, n_partial_rows - part_base);
        for (int64_t i = threadIdx.x; i < prows * hq * d; i += blockDim.x)
            part_o[part_base * hq * d + i] = __builtin_nanf("");
        for (int64_t i = threadIdx.x; i < prows * hq; i += blockDim.x)
            part_lse[part_base * hq + i] = __builtin_nanf("");
    }
}

// Key offset (within a 32-key block) held by register v of lane half h in
// the S^T accumulator, given the permuted K row order.
__device__ __forceinline__ int key_of_reg(int v, int h)
{
    return (v & 7) + 8 * h + 16 * (v >> 3);
}

// Permuted K row for MFMA row r: swap bits 2 and 3.
__device__ __forceinline__ int perm_row(int r)
{
    return (r & ~12) | ((r & 4) << 1) | ((r & 8) >> 1);
}

__device__ __forceinline__ float pair_max(float x)
{
    auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x),
                                              __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

__device__ __forceinline__ float pair_sum(float x)
{
    auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x),
                                              __float_as_uint(x), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Running maxima are re-based lazily: the output accumulator is rescaled only
// when a step's probabilities against the stale maximum could exceed this
// bound (2^8), so every probability stays at most 2^8.
constexpr float kRescaleBound = 256.0f;

typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

// LDS tiles hold 64 keys x D in the natural [key][d] order, rows of 2D bytes,
// with the 16-byte chunks of row r permuted by an XOR swizzle so that the
// MFMA operand reads are free of bank conflicts:
//   K (ds_read_b128 of 16 rows at one chunk): chunk' = chunk ^ kswz(r)
//   V (transposed ds_read_b64_tr_b16 of 4 rows x 4 chunks per 32 lanes):
//     chunk' = chunk ^ vswz(r)
template <int D>
__device__ __forceinline__ int kswz(int r)
{
    return D == 128 ? (r & 15) : ((r >> 1) & 7);
}
template <int D>
__device__ __forceinline__ int vswz(int r)
{
    return D == 128 ? 4 * (r & 3) : 4 * ((r >> 1) & 1);
}

// Trim an item's two runs of 64-key steps, [a_lo, a_hi) then [b_lo, b_hi),
// to the rows [wr0, wr_last] of one workgroup: steps whose keys all lie past
// its last row (causal), or, for streaming rows, outside the sink and before
// the window of its first row hold no kept pair and are skipped (their
// scores would all be masked, so the result is the same bit for bit).  The
// steps kept for streaming rows are those with a sink key, ceil(S / 64) from
// key 0, and those from the window start of the first row on.
__device__ __forceinline__ void trim_runs(bool stream, int sink, int window, int wr0,
                                          int wr_last, int &a_lo, int &a_hi, int &b_lo,
                                          int &b_hi)
{
    if (stream) {
        const int first = wr0 - window + 1;
        const int fs = first > 0 ? first / kStep : 0;  // first step with a window key
        const int ss = (sink + kStep - 1) / kStep;     // steps with a sink key
        if (b_hi > b_lo) {
            // run a holds the sink k-tiles, run b the band
            b_lo = min(max(b_lo, fs), b_hi);
            a_hi = max(min(a_hi, ss), a_lo);
        } else if (sink == 0) {
            a_lo = min(max(a_lo, fs), a_hi);
        } else if (fs > ss) {
            // one run holds the sink and the band: split off the keys between
            b_lo = min(fs, a_hi);
            b_hi = a_hi;
            a_hi = max(min(a_hi, ss), a_lo);
        }
    }
    const int ls = wr_last / kStep + 1;  // first step past the last row
    if (b_hi > b_lo)
        b_hi = max(min(b_hi, ls), b_lo);
    else
        a_hi = max(min(a_hi, ls), a_lo);
}

// Compile-time loop: f(std::integral_constant<int, I>) for I in [B, E).
template <int B, int E, typename F>
__device__ __forceinline__ void static_for(F &&f)
{
    if constexpr (B < E) {
        f(std::integral_constant<int, B>{});
        static_for<B + 1, E>(f);
    }
}

// LDS reads that MFMAs i .. i + count - 1 of a matrix phase need: one K
// fragment for each of the first NQ MFMAs (none for the first KPRE ones when
// they were read ahead), two transposed V reads for each later one.
template <int NQ, int N, int KPRE, bool PRE>
constexpr int phase_reads(int i, int count)
{
    int r = 0;
    for (int m = i; m < i + count && m < N; ++m)
        r += m >= NQ ? 2 : (PRE && m < KPRE) ? 0 : 1;
    return r;
}

// COPIER: the last of the NW waves only copies K/V tiles into LDS (all of
// them, at the start of each matrix phase of group 0) and computes nothing;
// the other NW - 1 waves compute.  For GQA group 7 (seven waves of 32 rows),
// whose eighth ping-pong slot would otherwise be empty: the MFMA waves then
// issue no copies.
// LIST: the kernel serves block-sparse schedules, whose list items read
// their k-tiles from the schedule's list section (the other kinds have none).
template <int D, int NW, bool COPIER = false, bool LIST = false>
__global__ __launch_bounds__(NW * 64, NW == 4 ? 2 : 1) void attn_tile_kernel(FwdArgs a,
                                                                               int32_t kind)
{
    constexpr int ROW_BYTES = 2 * D;
    constexpr int CHUNKS = D / 8;                       // 16-byte chunks per row
    constexpr int TILE_BYTES = kStep * ROW_BYTES;       // one K or V tile
    constexpr int STAGE_BYTES = 2 * TILE_BYTES;         // K tile, then V tile
    constexpr int N_STAGES = 2;                         // LDS double buffer
    constexpr int ROWS_PER_DMA = 1024 / ROW_BYTES;      // rows per wave copy
    constexpr int N_DMA = kStep / ROWS_PER_DMA;         // wave copies per tile
    // Only the waves of ping-pong group 0 copy K/V tiles into LDS, spread
    // over the MFMAs of their matrix phase (see the phase loop below), or
    // the copier wave alone.
    static_assert(!COPIER || NW == 8, "a copier wave beside seven compute waves");
    constexpr int NC = COPIER ? NW - 1 : NW;  // compute waves
    constexpr int N_COPY_WAVES = COPIER ? 1 : NW - NW / 2;
    constexpr int COPIES = (N_DMA + N_COPY_WAVES - 1) / N_COPY_WAVES;  // per tile
    constexpr int QK_STEPS = D / 16;
    constexpr int D_BLOCKS = D / 32;
    constexpr int MFMA_SLOTS = 2 * QK_STEPS + 4 * D_BLOCKS;  // MFMAs of a matrix phase
    constexpr int COPY_STRIDE = MFMA_SLOTS / (2 * COPIES) > 0
                                    ? MFMA_SLOTS / (2 * COPIES) : 1;

    // LDS: the two K/V stages, then one 32-row Q tile per wave (the prologue
    // stages Q there so that it is read from HBM in whole rows).  Workgroups
    // of at most four waves put their Q tiles in stage 1 instead, which
    // receives its first K/V copies only after every wave has read them:
    // their LDS then allows two workgroups per CU, and for four waves the
    // launch bound keeps them within 256 registers, so that every SIMD holds
    // two waves (the two of one workgroup's ping-pong pair sit on different
    // SIMDs).
    constexpr int QTILE_BYTES = 32 * ROW_BYTES;
    constexpr bool Q_IN_STAGE = NW * QTILE_BYTES <= STAGE_BYTES;
    constexpr int QREGION = Q_IN_STAGE ? STAGE_BYTES : N_STAGES * STAGE_BYTES;
    __shared__ __attribute__((aligned(1024))) unsigned char
        smem[N_STAGES * STAGE_BYTES + (Q_IN_STAGE ? 0 : NW * QTILE_BYTES)];
    static_assert(sizeof(smem) + (LIST ? kKeyTable * 4 : 0) <= 160 * 1024, "LDS of a CU");

    const int32_t *sched = a.sched;
    int bid = blockIdx.x;
    const int g = bid % a.hkv;
    bid /= a.hkv;
    const int sub = bid % a.subtiles;
    int item = bid / a.subtiles;
    if (item >= a.n_items)
        return;
    if (a.n_lead > 0) {
        // Launch slot x runs lead item floor(x n_lead / n_items) when that
        // count steps up at x, else the next of the other items: the lead
        // items (Last splits, each a run of k-tiles along the sequence) are
        // spread evenly through the launch, each beside the streaming q-tiles
        // whose bands have just read its keys into L2, instead of all reading
        // K and V from HBM at the start.  A bijection on [0, n_items).
        const uint32_t x = (uint32_t)item, nl = (uint32_t)a.n_lead, ni = (uint32_t)a.n_items;
        const uint32_t s0 = x * nl / ni, s1 = (x + 1) * nl / ni;
        item = s1 > s0 ? (int)s0 : (int)(nl + x - s1);
    }
    // The item words are read before the header is checked so that both
    // scalar loads are in flight together (the host has checked that the
    // schedule holds n_items items, so the read is in bounds either way).
    const int32_t *it = sched + kHdrWords + (int64_t)item * kItemWords;
    const int64_t seq_off = it[I_SEQ_OFF];
    const int32_t seq_len = it[I_SEQ_LEN];
    const int32_t r0 = it[I_R0], r1 = it[I_R1];
    const int32_t ka0 = it[I_KA0], ka1 = it[I_KA1];
    const int32_t kb0 = it[I_KB0], kb1 = it[I_KB1];
    const int32_t mode = it[I_MODE];
    const int32_t part_base = it[I_PART_BASE];
    // Guard against a schedule that does not match the launch, and against a
    // malformed item: never touch memory outside it; poison the outputs.
    // Block-sparse schedules record the length of their k-tile lists.  List
    // items (kModeCausalList) read the k-tiles list[ka0 .. ka0 + ka1) of the
    // tile-list section instead of two runs; only the list form of the kernel
    // accepts them, and no form accepts another mode.
    const bool list_mode = LIST && mode == kModeCausalList;
    // One combined test without short-circuits: the header and item words
    // are all loaded before it.
    const int32_t list_len = sched[H_WINDOW];  // block-sparse: length of the lists
    const bool bad =
        !header_ok(sched, a.total_tokens, a.n_items, kind) |
        (a.list_words != (kind == TA_KIND_BLOCKSPARSE ? list_len : 0)) |
        (seq_off < 0) | (seq_len < 0) | (seq_off + seq_len > a.total_tokens) | (r0 < 0) |
        (r1 > seq_len) | (r0 >= r1) | (ka0 < 0) | (kb0 < 0) | (kb1 < kb0) |
        (mode != kModeStreaming && mode != kModeCausal && !list_mode) |
        (list_mode ? (ka1 < 0) | (kb1 != kb0) | ((int64_t)ka0 + ka1 > a.list_words)
                   : ka1 < ka0) |
        ((part_base >= 0) & (part_base + (r1 - r0) > a.n_partial_rows));
    if (bad) {
        poison_outputs(a.o, a.o_f32, a.lse, a.total_tokens, a.hq, D, blockIdx.x,
                       gridDim.x);
        poison_item_rows(a.o, a.o_f32, a.lse, a.part_o, a.part_lse, a.total_tokens, a.hq, D,
                         a.n_partial_rows, a.tile, seq_off, r0, r1, part_base);
        return;
    }
    const int32_t *tile_list = sched + a.list_base + (list_mode ? ka0 : 0);
    const int max_ktile = seq_len > 0 ? (seq_len - 1) / a.tile : 0;

    const int wr0 = r0 + sub * a.rows_per_wg;  // first row of this workgroup
    if (wr0 >= r1)
        return;  // ragged q-tile: nothing for this workgroup

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    // The wave index is the same on every lane; reading it from lane 0 makes
    // everything derived from it (head, rows, ping-pong group) scalar, so the
    // per-wave branches below are uniform.
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int half = lane >> 5;
    const int col = lane & 31;
    const int waves_per_head = a.rows_per_wg / 32;
    const int head = g * a.group + wave / waves_per_head;
    const int row_base = wr0 + (wave % waves_per_head) * 32;
    const bool wave_active = row_base < r1;
    const int my_row = row_base + col;            // sequence-relative row
    const bool row_valid = my_row < r1;
    const int row_hi = (r1 - 1 < row_base + 31) ? r1 - 1 : row_base + 31;
    const float c = a.scale_log2;

    // Steps of 64 keys over the kept k-tiles: two runs, or a list (each
    // listed index clamped to the sequence's k-tiles).  The runs are trimmed
    // to this workgroup's rows (trim_runs).
    const int tps = a.tile / kStep;
    const int wr_last = min(wr0 + a.rows_per_wg, r1) - 1;
    int a_lo = ka0 * tps, a_hi = ka1 * tps, b_lo = kb0 * tps, b_hi = kb1 * tps;
    if (!list_mode)
        trim_runs(mode == kModeStreaming, a.sink, a.window, wr0, wr_last, a_lo, a_hi, b_lo,
                  b_hi);
    const int na = list_mode ? ka1 * tps : a_hi - a_lo;
    int nsteps = list_mode ? na : na + (b_hi - b_lo);
    // A list item's step keys are read from the list once, into an LDS
    // table, so that no step waits on a global load (a global load's wait
    // would also wait for the K/V copies in flight).  Longer lists than the
    // table read the list at every step.
    typedef __attribute__((address_space(3))) int32_t lds_i32;
    lds_i32 *keytab = nullptr;
    if constexpr (LIST) {
        __shared__ int32_t tab[kKeyTable];
        keytab = (lds_i32 *)tab;
    }
    const bool use_tab = list_mode && na <= kKeyTable;
    if (use_tab) {
        for (int s = threadIdx.x; s < na; s += NW * 64) {
            const int kt = min(max(tile_list[s / tps], 0), max_ktile);
            keytab[s] = kt * a.tile + (s % tps) * kStep;
        }
        __syncthreads();
    }
    auto step_key0 = [&](int s) TA_INLINE -> int {
        if (list_mode) {
            if (use_tab)
                return keytab[s];
            const int kt = min(max(tile_list[s / tps], 0), max_ktile);
            return kt * a.tile + (s % tps) * kStep;
        }
        return s < na ? (a_lo + s) * kStep : (b_lo + (s - na)) * kStep;
    };
    if (list_mode)  // listed tiles increase: only the last may pass the rows
        while (nsteps > 0 && step_key0(nsteps - 1) > wr_last)
            --nsteps;

    // Q fragments (B operand of S^T = K Q^T): lane holds Q[row][16s + 8h ..].
    // The wave's 32 Q rows are first copied whole into its LDS Q tile (1 KB
    // per copy = 1024 / ROW_BYTES rows; lane l lands at byte 16 l: row
    // l / CHUNKS of the copy, stored chunk l % CHUNKS holding logical chunk
    // (l % CHUNKS) ^ kswz(row)), then read in fragment order after the
    // prologue barrier.  Rows past the q-tile repeat its last row.
    const uint32_t smem_addr =
        (uint32_t)(uintptr_t)(__attribute__((address_space(3))) void *)smem;
    const int q_row0 = min(row_base, r1 - 1);  // the wave's first row to read
    if (!COPIER || wave < NC) {
        const uint16_t *qb = a.q + ((seq_off + q_row0) * a.hq + head) * (int64_t)D;
        const uint32_t q_pitch = (uint32_t)(a.hq * ROW_BYTES);
#pragma unroll
        for (int i = 0; i < QTILE_BYTES / 1024; ++i) {
            const int row = i * (1024 / ROW_BYTES) + lane / CHUNKS;
            const int rr = min(row_base + row, r1 - 1) - q_row0;  // 0 .. 31
            const uint32_t off = __umul24((uint32_t)rr, q_pitch) +
                                 (uint32_t)(((lane % CHUNKS) ^ kswz<D>(row)) << 4);
            copy_to_lds16(qb, off, smem_addr + QREGION + wave * QTILE_BYTES + i * 1024);
        }
    }
    bf16x8 qf[QK_STEPS];
    auto read_q = [&]() TA_INLINE {
        const unsigned char *qt = smem + QREGION + wave * QTILE_BYTES + col * ROW_BYTES;
#pragma unroll
        for (int s = 0; s < QK_STEPS; ++s)
            qf[s] = *reinterpret_cast<const bf16x8 *>(qt + (((2 * s + half) ^ kswz<D>(col)) << 4));
    };

    const uint16_t *kbase = a.k + (seq_off * a.hkv + g) * (int64_t)D;
    const uint16_t *vbase = a.v + (seq_off * a.hkv + g) * (int64_t)D;
    const int tok_stride = a.hkv * D;

    // Global -> LDS copies: copy number m of a tile writes 1 KB = ROWS_PER_DMA
    // rows; lane l lands at byte 16 l of it, i.e. row m*ROWS_PER_DMA +
    // l / CHUNKS, stored chunk l % CHUNKS, which holds logical chunk
    // (l % CHUNKS) ^ swizzle(row).  Copy waves (group 0, wave w < N_COPY_WAVES)
    // own copies m = w, w + N_COPY_WAVES, ... of every K and V tile.
    const bool copy_wave = COPIER ? wave == NW - 1 : wave < N_COPY_WAVES;
    const int copy_rank = COPIER ? 0 : wave;  // the wave's first copy number
    const int dma_row_in = lane / CHUNKS;
    const int dma_pc = lane % CHUNKS;
    // The swizzle of row m * ROWS_PER_DMA + i is swizzle(i) ^ swizzle of the
    // copy's first row (K) or swizzle(i) (V): the copy's first row is a
    // multiple of ROWS_PER_DMA, whose swizzle bits lie above those of i.
    const uint32_t kx0 = (uint32_t)((dma_pc ^ kswz<D>(dma_row_in)) << 4);
    const uint32_t vx0 = (uint32_t)((dma_pc ^ vswz<D>(dma_row_in)) << 4);
    const uint32_t row_stride_bytes = 2u * (uint32_t)tok_stride;  // < 2^24 (host check)
    // Byte offset of the row of the tile that this lane copies in the wave's
    // first copy, and the step from one of the wave's copies to the next.
    const uint32_t dma_off0 =
        __umul24((uint32_t)(copy_rank * ROWS_PER_DMA + dma_row_in), row_stride_bytes);
    const uint32_t dma_off_step = (uint32_t)(N_COPY_WAVES * ROWS_PER_DMA) * row_stride_bytes;
    // The K swizzle term of copy i, kswz((wave + i * N_COPY_WAVES) *
    // ROWS_PER_DMA), does not depend on i when N_COPY_WAVES * ROWS_PER_DMA
    // is a multiple of the swizzle period (16 rows for d = 128, 8 rows of
    // bit 1..3 for d = 64): then one clamp bound per tile serves every copy.
    constexpr bool XR_PER_WAVE = D == 128 ? N_COPY_WAVES % 4 == 0 : N_COPY_WAVES % 2 == 0;
    // Keys past the end of the sequence are read from its last row: they lie
    // beyond every row of the item, so the causal mask gives them p = 0.
    const int key_max = seq_len - 1;

    // One tile copy (K or V of one step into one stage).  Row r of the tile
    // reads key min(key0 + r, last key of the sequence), so a step past the
    // end of the sequence still reads valid rows.  The scalar base is the
    // tile's first key kc = min(key0, last key); lane row r adds the byte
    // offset min(r, last key - kc) * row pitch (the clamp is taken on the
    // byte offsets, which are monotonic in r), an unsigned 32-bit offset of
    // fewer than 64 rows that is never negative.  Everything that depends
    // only on the tile is computed once here, so a copy costs one M0 write,
    // a nop, the clamp and the copy itself.  Workgroups whose tiles all lie
    // inside the sequence use the burst form instead (BURST below: no clamp,
    // one M0 write per four copies).
    struct TileCopy {
        const uint16_t *base;  // row kc of the source
        uint32_t lds;          // LDS address of this wave's first copy
        uint32_t lim;          // min(last key - kc, 63) * row pitch in bytes
    };
    auto plan_copy = [&](const uint16_t *src, int key0, int buf,
                         bool is_v) TA_INLINE -> TileCopy {
        // key0 is the same on every lane (it may come from the LDS key table)
        const int kc = __builtin_amdgcn_readfirstlane(min(key0, key_max));
        TileCopy t;
        t.base = src + (int64_t)kc * tok_stride;
        t.lim = (uint32_t)min(key_max - kc, kStep - 1) * row_stride_bytes;
        t.lds = smem_addr + buf * STAGE_BYTES + (is_v ? TILE_BYTES : 0) + copy_rank * 1024;
        return t;
    };
    // Copy i of this wave (m = copy_rank + i * N_COPY_WAVES) of a planned tile.
    auto issue_copy = [&](const TileCopy &t, int i, bool is_v) TA_INLINE {
        const int m = copy_rank + i * N_COPY_WAVES;
        if constexpr (N_DMA % N_COPY_WAVES != 0) {
            if (m >= N_DMA)
                return;
        }
        const uint32_t xr = is_v ? vx0 : (kx0 ^ (uint32_t)(kswz<D>(m * ROWS_PER_DMA) << 4));
        uint32_t off;
        if constexpr (XR_PER_WAVE) {
            // min(r, lim) + xr = min(r + xr, lim + xr): the first term is a
            // constant of the lane and copy, the second of the lane and tile
            off = min(dma_off0 + (uint32_t)i * dma_off_step + xr, t.lim + xr);
        } else {
            off = min(dma_off0 + (uint32_t)i * dma_off_step, t.lim) + xr;
        }
        copy_to_lds16(t.base, off, t.lds + i * (N_COPY_WAVES * 1024));
    };
    // Copy slot c (0 <= c < 2 * COPIES): K copies first, then V copies.
    TileCopy cp_k{}, cp_v{};
    auto issue_slot = [&](int c) TA_INLINE {
        if (c < COPIES)
            issue_copy(cp_k, c, false);
        else
            issue_copy(cp_v, c - COPIES, true);
    };
    // Hook run after MFMA number `slot` of a matrix phase of a copy wave.
    auto copy_hook = [&](int slot) TA_INLINE {
        if (slot % COPY_STRIDE == COPY_STRIDE - 1 && slot / COPY_STRIDE < 2 * COPIES)
            issue_slot(slot / COPY_STRIDE);
    };
    auto no_hook = [](int) {};
    // The hook of group 0's matrix phases: its copies, unless a copier wave
    // makes them.
    auto g0_hook = [&](int slot) TA_INLINE {
        if constexpr (!COPIER)
            copy_hook(slot);
    };
    // Burst form of group 0's copies, for workgroups whose K/V tiles all lie
    // inside the sequence (nothing to clamp): copy wave w copies the
    // consecutive 1 KB blocks w * COPIES .. w * COPIES + COPIES - 1 of a
    // tile in one burst with one M0 write, K after the copy slot of the first
    // K copy and V after that of the first V copy.  Its lane offsets are
    // constants of the lane (row * pitch + swizzled chunk - i KB, i the
    // block's index in the burst, which the instruction offset adds back).
    constexpr bool BURST =
        !COPIER && (COPIES == 2 || COPIES == 4) && N_DMA == COPIES * N_COPY_WAVES;
    constexpr int BURST_K_SLOT = COPY_STRIDE - 1;
    constexpr int BURST_V_SLOT = COPIES * COPY_STRIDE + COPY_STRIDE - 1;
    // from a planned copy's LDS address (block copy_rank of the tile) to the
    // first block of this wave's burst (block copy_rank * COPIES)
    const uint32_t burst_lds = (uint32_t)(copy_rank * (COPIES - 1) * 1024);

    // S^T = K Q^T for one 64-key step from LDS stage `buf`; the two 32-key
    // accumulator chains alternate so that dependent MFMAs do not stall.
    // K fragment (kb, s): row kb * 32 + perm_row(col), chunk (2s + half) ^
    // kswz(row); the swizzle does not depend on kb, so one offset per s.
    const int krow0 = perm_row(col);
    uint32_t koff[QK_STEPS];
#pragma unroll
    for (int s = 0; s < QK_STEPS; ++s)
        koff[s] = (uint32_t)(krow0 * ROW_BYTES + (((2 * s + half) ^ kswz<D>(krow0)) << 4));
    // The first KPRE K fragments of a matrix phase can be read ahead, in the
    // wave's softmax phase before it, when the stage has landed by then: the
    // first MFMAs of the phase then wait for no LDS read.
    constexpr int KPRE = 2 * QK_STEPS < 6 ? 2 * QK_STEPS : 6;
    bf16x8 kpre[KPRE];
    auto prefetch_k = [&](int buf) TA_INLINE {
        const unsigned char *kt = smem + buf * STAGE_BYTES;
#pragma unroll
        for (int i = 0; i < KPRE; ++i)
            kpre[i] = *reinterpret_cast<const bf16x8 *>(kt + koff[i / 2] +
                                                          (i & 1) * 32 * ROW_BYTES);
    };
    auto qk = [&](int buf, f32x16 (&sacc)[2], auto hook, auto pre, auto own) TA_INLINE {
        constexpr bool PRE = decltype(pre)::value;
        const unsigned char *kt = smem + buf * STAGE_BYTES;
        sacc[0] = f32x16{};
        sacc[1] = f32x16{};
#pragma unroll
        for (int s = 0; s < QK_STEPS; ++s) {
            bf16x8 a0, a1;
            if (PRE && 2 * s + 1 < KPRE) {
                a0 = kpre[2 * s];
                a1 = kpre[2 * s + 1];
            } else {
                a0 = *reinterpret_cast<const bf16x8 *>(kt + koff[s]);
                a1 = *reinterpret_cast<const bf16x8 *>(kt + koff[s] + 32 * ROW_BYTES);
            }
            sacc[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, qf[s], sacc[0], 0, 0, 0);
            hook(2 * s);
            sacc[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, qf[s], sacc[1], 0, 0, 0);
            hook(2 * s + 1);
        }
        constexpr int n = 2 * QK_STEPS, ahead = 6;
        if constexpr (!decltype(own)::value) {
            // the caller schedules the reads of the whole phase
        } else if constexpr (PRE) {
            // read r feeds MFMA KPRE + r: one read before each MFMA from the
            // first keeps them KPRE MFMAs ahead
#pragma unroll
            for (int i = 0; i < n - KPRE; ++i) {
                __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 1, 0);
                __builtin_amdgcn_sched_group_barrier(kSchedMfma, 1, 0);
            }
            __builtin_amdgcn_sched_group_barrier(kSchedMfma, KPRE, 0);
        } else {
            // keep six operand reads in flight ahead of the MFMAs
            __builtin_amdgcn_sched_group_barrier(kSchedDsRead, ahead, 0);
#pragma unroll
            for (int i = 0; i < n - ahead; ++i) {
                __builtin_amdgcn_sched_group_barrier(kSchedMfma, 1, 0);
                __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 1, 0);
            }
            __builtin_amdgcn_sched_group_barrier(kSchedMfma, ahead, 0);
        }
    };

    f32x16 oacc[D_BLOCKS];
#pragma unroll
    for (int b = 0; b < D_BLOCKS; ++b)
        oacc[b] = f32x16{};

    // O^T += V^T P^T for one 64-key step from LDS stage `buf`.  The V^T
    // fragment of 8 keys x 1 d comes from two transposed reads: in each group
    // of 16 lanes, lane i addresses row K0 + i/4 at d = D0 + 4 (i % 4), and
    // lane j receives rows K0..K0+3 at d = D0 + j.
    // Rows differ from 8 half + i/4 by multiples of 4, which leave the V
    // swizzle unchanged, so one offset per d block plus an immediate covers
    // every read.
    const int vrow0 = 8 * half + ((lane & 15) >> 2);
    const int tr_d = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);  // + 32 b
    uint32_t voff[D_BLOCKS];
#pragma unroll
    for (int b = 0; b < D_BLOCKS; ++b) {
        const int d = 32 * b + tr_d;
        voff[b] = (uint32_t)(vrow0 * ROW_BYTES + (((d >> 3) ^ vswz<D>(vrow0)) << 4) +
                             (d & 7) * 2);
    }
    auto pv = [&](int buf, const bf16x8 (&pf)[2][2], auto hook, auto own) TA_INLINE {
        const unsigned char *vt = smem + buf * STAGE_BYTES + TILE_BYTES;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
            for (int s2 = 0; s2 < 2; ++s2)
#pragma unroll
                for (int b = 0; b < D_BLOCKS; ++b) {
                    s16x4 part[2];
#pragma unroll
                    for (int i2 = 0; i2 < 2; ++i2)
                        part[i2] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                            (lds_s16x4 *)(vt + voff[b] +
                                          (kb * 32 + s2 * 16 + 4 * i2) * ROW_BYTES));
                    const bf16x8 af = __builtin_bit_cast(
                        bf16x8, __builtin_shufflevector(part[0], part[1], 0, 1, 2, 3, 4, 5,
                                                        6, 7));
                    oacc[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af, pf[kb][s2],
                                                                     oacc[b], 0, 0, 0);
                    hook(2 * QK_STEPS + (kb * 2 + s2) * D_BLOCKS + b);
                }
        // two transposed reads per MFMA; keep four MFMAs' operands in flight
        if constexpr (decltype(own)::value) {
            constexpr int n = 4 * D_BLOCKS, ahead = 4;
            __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 2 * ahead, 0);
#pragma unroll
            for (int i = 0; i < n - ahead; ++i) {
                __builtin_amdgcn_sched_group_barrier(kSchedMfma, 1, 0);
                __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 2, 0);
            }
            __builtin_amdgcn_sched_group_barrier(kSchedMfma, ahead, 0);
        }
    };
    // Reads of a whole matrix phase (QK^T then PV) in one sequence: MFMA i
    // needs one K read (i < NQ, none for prefetched fragments) or two V
    // reads; the reads of MFMA i + ahead are issued just before MFMA i, so
    // the first V reads overlap the last QK^T MFMAs instead of waiting for
    // them to issue.
    auto sched_phase = [&](auto pre) TA_INLINE {
        constexpr bool PRE = decltype(pre)::value;
        constexpr int NQ = 2 * QK_STEPS, N = NQ + 4 * D_BLOCKS, ahead = 6;
        constexpr int first = phase_reads<NQ, N, KPRE, PRE>(0, ahead);
        if constexpr (first > 0)
            __builtin_amdgcn_sched_group_barrier(kSchedDsRead, first, 0);
        static_for<0, N>([&](auto ic) TA_INLINE {
            constexpr int nr = phase_reads<NQ, N, KPRE, PRE>(decltype(ic)::value + ahead, 1);
            __builtin_amdgcn_sched_group_barrier(kSchedMfma, 1, 0);
            if constexpr (nr > 0)
                __builtin_amdgcn_sched_group_barrier(kSchedDsRead, nr, 0);
        });
    };

    // Element mask (branch-free selects) where the step crosses the diagonal
    // or the window edge; keys beyond the sequence are beyond every row.  The
    // cases are told apart per wave, so that a step needs one compare per
    // score where only one bound applies: the causal bound on the diagonal,
    // the sink bound on a step before every row's window, the window bound
    // at the window edge; both only where a step holds more than one edge.
    auto mask_step = [&](int key0, bool need_causal, bool need_window,
                         f32x16 (&sacc)[2]) TA_INLINE {
        const int lim = my_row - key0 - 8 * half;  // key offset <= lim: causal
        if (!need_window) {
            // every key is a sink key or inside every row's window
            if (need_causal) {
#pragma unroll
                for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                    for (int v = 0; v < 16; ++v) {
                        const int off = kb * 32 + key_of_reg(v, 0);
                        sacc[kb][v] = off <= lim ? sacc[kb][v] : -INFINITY;
                    }
            }
            return;
        }
        const int win_lim = lim - a.window;             // offset > win_lim: in the window
        const int sink_lim = a.sink - key0 - 8 * half;  // offset < sink_lim: a sink key
        if (key0 + kStep - 1 <= row_base - a.window) {
            // before every row's window (and diagonal): only sink keys remain
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int off = kb * 32 + key_of_reg(v, 0);
                    sacc[kb][v] = off < sink_lim ? sacc[kb][v] : -INFINITY;
                }
            return;
        }
        if (!need_causal && key0 >= a.sink) {
            // past the sink and before every row's diagonal: the window edge
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int off = kb * 32 + key_of_reg(v, 0);
                    sacc[kb][v] = off > win_lim ? sacc[kb][v] : -INFINITY;
                }
            return;
        }
        // several bounds: sign-bit masks (all ones where kept) in vector
        // registers, combined and applied with bit operations.  The score is
        // copied out of the vector before its bits are taken: a bit cast of
        // a vector element itself compiles to a read of element 0.
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int off = kb * 32 + key_of_reg(v, 0);  // 8 half is in lim
                const int m = ~((lim - off) >> 31) &
                              (((off - sink_lim) >> 31) | ((win_lim - off) >> 31));
                const float sc = sacc[kb][v];
                sacc[kb][v] = __builtin_bit_cast(
                    float, (__builtin_bit_cast(uint32_t, sc) & (uint32_t)m) |
                               (0xff800000u & ~(uint32_t)m));
            }
    };

    float m_ref = -INFINITY;  // reference maximum of the row, log2 domain
    // the maximum the probabilities are taken against: m_ref once set; while
    // it is -inf, a plain pass yields an infinite or NaN sum, which sends the
    // step to the re-base as an unset maximum must
    float m_cur = -INFINITY;
    float l_run = 0.f;        // running sum over this lane's keys
    bool fresh = true;        // the first softmax: no reference maximum on any lane

    // Online softmax of one step: probabilities relative to the (lazily
    // re-based) reference maximum, converted to the bf16 B operand of PV.
    // O holds every earlier step already, so a re-base rescales it here.
    // The probabilities are first taken against the current reference: each
    // is >= 0, so if their sum is at most kRescaleBound none exceeds it and
    // the step needs no row maximum at all.  Only when the sum is larger (a
    // maximum has grown by up to log2(kRescaleBound) powers of two or more)
    // or no reference is set yet does the wave compute the row maxima,
    // re-base to them and redo the step.  Either way every probability that
    // enters O and l is at most kRescaleBound and the row maximum itself,
    // once seen, contributes at least 1 (no underflow of l).
    auto softmax = [&](f32x16 (&sacc)[2], bf16x8 (&pf)[2][2]) TA_INLINE {
        auto exp_step = [&](float m_use) TA_INLINE -> float {
            float psum = 0.f;
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int s2 = 0; s2 < 2; ++s2) {
                    f32x8 t;
#pragma unroll
                    for (int e = 0; e < 8; ++e) {
                        t[e] = __builtin_amdgcn_exp2f(
                            __builtin_fmaf(sacc[kb][8 * s2 + e], c, -m_use));
                        // the sum starts at the first term (exp2 is never -0)
                        psum = (kb | s2 | e) ? psum + t[e] : t[e];
                    }
                    pf[kb][s2] = __builtin_convertvector(t, bf16x8);
                }
            return psum;
        };
        // The first step has no reference on any lane: it goes straight to
        // the re-base (its first pass would be discarded).
        float psum = INFINITY;
        if (!fresh)
            psum = exp_step(m_cur);
        fresh = false;
        const bool bad = !(psum <= kRescaleBound);
        if (__builtin_amdgcn_ballot_w64(bad) != 0) {
            float mx = -INFINITY;
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int v = 0; v < 16; ++v)
                    mx = fmaxf(mx, sacc[kb][v]);
            mx = pair_max(mx);
            const float m_new = fmaxf(m_ref, mx * c);
            const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
            const float alpha = __builtin_amdgcn_exp2f(m_ref - m_use);
            l_run *= alpha;
#pragma unroll
            for (int b = 0; b < D_BLOCKS; ++b)
                oacc[b] *= alpha;
            m_ref = m_new;
            m_cur = m_new;
            psum = exp_step(m_use);
        }
        l_run += psum;
    };

    // Two-group ping-pong.  The waves are split into two groups with one wave
    // of each group on every SIMD.  Work of a wave, in order: M(0), X(0),
    // M(1), X(1), ..., M(n), where M(j) = { S(j) = K(j) Q^T ; O += V(j-1)
    // P(j-1) } runs on the matrix cores and X(j) = softmax of S(j) runs on
    // the vector units.  Group 0 runs M(j) in phase 2j and X(j) in phase
    // 2j + 1; group 1 runs X(j-1) in phase 2j and M(j) in phase 2j + 1, so in
    // every phase one wave of each SIMD issues MFMAs while the other issues
    // the softmax.  LDS stage j & 1 holds K(j) and V(j-1) for phases 2j and
    // 2j+1.  During M(j) the group-0 waves copy K(j+1) and V(j) into stage
    // (j+1) & 1 (last read in phase 2j-1), one copy after every COPY_STRIDE
    // MFMAs so that the address units see a steady stream, and wait for them
    // at the end of phase 2j+1.  The softmax waves issue no copies.  With a
    // copier wave (seven compute waves: four in group 0, three in group 1),
    // that wave makes all of these copies and group 0 none.
    const int n_group1 = NW / 2;  // the copier wave, if any, returns before
    const int group = NW >= 2 ? (wave >= NW - n_group1 ? 1 : 0) : 0;
    f32x16 s_acc[2];
    bf16x8 p_acc[2][2];

    // Matrix phase: QK^T of step j (if any) and PV of step j-1 (if any).
    // Inside the step loops (unrolled by two) the LDS stage is a
    // std::integral_constant, so every LDS operand address is a per-lane
    // offset plus an immediate.
    // prep() runs inside the phase, so that its scalar work (planning the
    // phase's copies) can overlap the first LDS reads.
    auto no_prep = []() {};
    auto do_m = [&](auto stage, bool has_qk, bool has_pv, auto hook, auto pre,
                    auto prep) TA_INLINE {
        __builtin_amdgcn_sched_barrier(0);
        __builtin_amdgcn_s_setprio(1);  // MFMA issue goes first on the SIMD
        __builtin_amdgcn_sched_barrier(0);
        prep();
        const int buf = stage;
        if (!COPIER && has_qk && has_pv) {
            qk(buf, s_acc, hook, pre, std::false_type{});
            pv(buf, p_acc, hook, std::false_type{});
            sched_phase(pre);
        } else {
            if (has_qk)
                qk(buf, s_acc, hook, pre, std::true_type{});
            if (has_pv)
                pv(buf, p_acc, hook, std::true_type{});
        }
        __builtin_amdgcn_sched_barrier(0);
        __builtin_amdgcn_s_setprio(0);
        __builtin_amdgcn_sched_barrier(0);
    };
    auto do_x = [&](int j) TA_INLINE {
        const int key0 = step_key0(j);
        // the step crosses its rows' diagonal, or a window edge
        const bool need_causal = key0 + kStep - 1 > row_base;
        const bool need_window = mode == kModeStreaming && key0 + kStep - 1 >= a.sink &&
                                 row_hi - key0 >= a.window;
        if (__builtin_expect(need_causal | need_window, 0))  // a few steps per item
            mask_step(key0, need_causal, need_window, s_acc);
        softmax(s_acc, p_acc);
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
            for (int s2 = 0; s2 < 2; ++s2)
                fence_regs(p_acc[kb][s2]);
        fence_regs(l_run);
        fence_regs(m_ref);
        fence_regs(m_cur);
    };
    // A phase boundary: the scheduler may not move any instruction across it
    // (MFMAs and VALU work must stay in their own phase).
    auto end_phase = [&](bool wait_copies) TA_INLINE {
        __builtin_amdgcn_sched_barrier(0);
        if (wait_copies)
            wait_vmcnt(0);
        barrier_no_fence();
        __builtin_amdgcn_sched_barrier(0);
    };
    // Copies of K(j+1) and V(j) into stage (j+1) & 1 (clamped sources: copies
    // for steps past the last one land in parts of the stage nobody reads).
    auto plan_step_copies = [&](int j, auto stage) TA_INLINE {
        const int nbuf = 1 - (int)stage;  // stage (j + 1) & 1
        cp_k = plan_copy(kbase, step_key0(min(j + 1, nsteps - 1)), nbuf, false);
        cp_v = plan_copy(vbase, step_key0(min(j, nsteps - 1)), nbuf, true);
    };
    using Stage0 = std::integral_constant<int, 0>;
    using Stage1 = std::integral_constant<int, 1>;

    if constexpr (COPIER) {
        // The copier wave: K(0) in the prologue, then for every step j the
        // copies of K(j+1) and V(j) at the start of phase 2j, waited for at
        // the end of phase 2j+1; its barriers match those of the other waves.
        if (wave == NW - 1) {
            if (nsteps > 0) {
                cp_k = plan_copy(kbase, step_key0(0), 0, false);
#pragma unroll
                for (int c = 0; c < COPIES; ++c)
                    issue_slot(c);
                end_phase(true);
                if constexpr (Q_IN_STAGE)
                    end_phase(false);
                // When every tile lies inside the sequence (the steps' keys
                // increase, so when the last one does), the copies go out in
                // bursts of four consecutive 1 KB blocks: one M0 write per
                // burst, the blocks placed by the instruction offset, and the
                // burst's rows reached through the scalar base, so that four
                // lane offsets per tensor serve every burst.
                if (step_key0(nsteps - 1) + kStep - 1 <= key_max) {
                    constexpr int GROUP_ROWS = 4 * ROWS_PER_DMA;
                    static_assert(N_DMA % 4 == 0, "whole bursts of four copies");
                    uint32_t bk[4], bv[4];
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const int row = i * ROWS_PER_DMA + dma_row_in;
                        const uint32_t ro = __umul24((uint32_t)row, row_stride_bytes) -
                                            (uint32_t)(i * 1024);
                        bk[i] = ro + (uint32_t)((dma_pc ^ kswz<D>(row)) << 4);
                        bv[i] = ro + (uint32_t)((dma_pc ^ vswz<D>(row)) << 4);
                    }
                    for (int j = 0; j < nsteps; ++j) {
                        plan_step_copies(j, j & 1);
#pragma unroll
                        for (int g4 = 0; g4 < N_DMA / 4; ++g4)
                            copy_burst_to_lds16<4>(cp_k.base + g4 * GROUP_ROWS * tok_stride, bk,
                                                   cp_k.lds + g4 * 4096);
#pragma unroll
                        for (int g4 = 0; g4 < N_DMA / 4; ++g4)
                            copy_burst_to_lds16<4>(cp_v.base + g4 * GROUP_ROWS * tok_stride, bv,
                                                   cp_v.lds + g4 * 4096);
                        end_phase(false);
                        end_phase(true);
                    }
                } else {
                    for (int j = 0; j < nsteps; ++j) {
                        plan_step_copies(j, j & 1);
#pragma unroll
                        for (int c = 0; c < 2 * COPIES; ++c)
                            issue_slot(c);
                        end_phase(false);
                        end_phase(true);
                    }
                }
                end_phase(false);
                end_phase(false);
            }
            return;
        }
    }
    if (nsteps > 0) {
        // Prologue: the copy waves copy K(0) into stage 0.
        if (copy_wave) {
            cp_k = plan_copy(kbase, step_key0(0), 0, false);
#pragma unroll
            for (int c = 0; c < COPIES; ++c)
                issue_slot(c);
        }
        end_phase(true);  // K(0) and every wave's Q tile have landed
        read_q();
        if constexpr (Q_IN_STAGE)
            end_phase(false);  // stage 1 is free once every wave has read its Q
        if (group == 0) {
            auto run_group0 = [&](auto burst) TA_INLINE {
                constexpr bool B = decltype(burst)::value;
                uint32_t bk[B ? COPIES : 1], bv[B ? COPIES : 1];
                if constexpr (B) {
#pragma unroll
                    for (int i = 0; i < COPIES; ++i) {
                        // row >= i * ROWS_PER_DMA rows of at least 1024 / ROWS_PER_DMA
                        // bytes each, so subtracting i KB cannot wrap
                        const int row = (copy_rank * COPIES + i) * ROWS_PER_DMA + dma_row_in;
                        const uint32_t ro = __umul24((uint32_t)row, row_stride_bytes) -
                                            (uint32_t)(i * 1024);
                        bk[i] = ro + (uint32_t)((dma_pc ^ kswz<D>(row)) << 4);
                        bv[i] = ro + (uint32_t)((dma_pc ^ vswz<D>(row)) << 4);
                    }
                }
                auto burst_k = [&]() TA_INLINE {
                    if constexpr (B)
                        copy_burst_to_lds16<COPIES>(cp_k.base, bk, cp_k.lds + burst_lds);
                };
                auto burst_v = [&]() TA_INLINE {
                    if constexpr (B)
                        copy_burst_to_lds16<COPIES>(cp_v.base, bv, cp_v.lds + burst_lds);
                };
                auto hook = [&](int slot) TA_INLINE {
                    if constexpr (B) {
                        if (slot == BURST_K_SLOT)
                            burst_k();
                        else if (slot == BURST_V_SLOT)
                            burst_v();
                    } else {
                        g0_hook(slot);
                    }
                };
                // j = 0: QK only, then the copies of the PV slots.
                auto prep0 = [&]() TA_INLINE {
                    if constexpr (!COPIER)
                        plan_step_copies(0, Stage0{});
                };
                do_m(Stage0{}, true, false, hook, std::false_type{}, prep0);
                if constexpr (B) {
                    if constexpr (BURST_V_SLOT >= 2 * QK_STEPS)
                        burst_v();
                } else if constexpr (!COPIER) {
#pragma unroll
                    for (int c = 0; c < 2 * COPIES; ++c)
                        if (c * COPY_STRIDE + COPY_STRIDE - 1 >= 2 * QK_STEPS)
                            issue_slot(c);
                }
                end_phase(false);
                do_x(0);
                end_phase(true);
                // step j reads stage j & 1 (odd j first)
                auto step = [&](int j, auto stage) TA_INLINE {
                    auto prep = [&]() TA_INLINE {
                        if constexpr (!COPIER)
                            plan_step_copies(j, stage);
                    };
                    do_m(stage, true, true, hook, std::false_type{}, prep);
                    end_phase(false);
                    do_x(j);
                    end_phase(true);
                };
                int j = 1;
                for (; j + 1 < nsteps; j += 2) {
                    step(j, Stage1{});
                    step(j + 1, Stage0{});
                }
                if (j < nsteps)
                    step(j, Stage1{});
                do_m(nsteps & 1, false, true, no_hook, std::false_type{}, no_prep);
                end_phase(false);
                end_phase(false);
            };
            // The steps' keys increase, so every tile lies inside the
            // sequence when the last step's does (the copies past the last
            // step repeat it).
            if constexpr (BURST) {
                if (step_key0(nsteps - 1) + kStep - 1 <= key_max)
                    run_group0(std::true_type{});
                else
                    run_group0(std::false_type{});
            } else {
                run_group0(std::false_type{});
            }
        } else {
            // Group 1's matrix phase M(j) reads stage j & 1, whose K(j) has
            // landed before the phase in which group 1 runs X(j - 1): the
            // first K fragments of M(j) are read at the start of that phase
            // (not with a copier wave, where it measured slower).
            constexpr bool PRE = !COPIER;
            if constexpr (PRE)
                prefetch_k(0);
            end_phase(false);
            do_m(Stage0{}, true, false, no_hook, std::bool_constant<PRE>{}, no_prep);
            end_phase(false);
            auto step = [&](int j, auto stage) TA_INLINE {
                if constexpr (PRE)
                    prefetch_k(stage);
                do_x(j - 1);
                end_phase(false);
                do_m(stage, true, true, no_hook, std::bool_constant<PRE>{}, no_prep);
                end_phase(false);
            };
            int j = 1;
            for (; j + 1 < nsteps; j += 2) {
                step(j, Stage1{});
                step(j + 1, Stage0{});
            }
            if (j < nsteps)
                step(j, Stage1{});
            do_x(nsteps - 1);
            end_phase(false);
            do_m(nsteps & 1, false, true, no_hook, std::false_type{}, no_prep);
            end_phase(false);
        }
    } else {
        wait_vmcnt(0);  // no steps: the Q copies must still land before exit
    }

    if (!wave_active)
        return;
    const float l_tot = pair_sum(l_run);
    const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
    const float row_lse = l_tot > 0.f ? (m_ref + __log2f(l_tot)) * kLn2 : -INFINITY;

    if (part_base < 0 && !a.o_f32) {
        // bf16 output rows, written whole: a lane holds 4-value pieces of
        // its row spread over the row, so the wave first stages its 32 x D
        // tile in its own slice of the (now idle) K/V stages, XOR-swizzled
        // by 16-byte chunk, then stores complete rows.  Every wave has
        // passed the last barrier of the loop, after which no LDS read or
        // copy of the loop is outstanding.
        constexpr int ROWB = D * 2;    // bytes per output row
        constexpr int CHK = ROWB / 16; // 16-byte chunks per row
        static_assert(NW * 32 * ROWB <= N_STAGES * STAGE_BYTES, "epilogue tile fits the stages");
        unsigned char *tile = smem + wave * (32 * ROWB);
        auto oswz = [](int r) { return D == 128 ? (r & 15) : ((r >> 1) & 7); };
#pragma unroll
        for (int b = 0; b < D_BLOCKS; ++b)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                f32x4 t;
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    t[e] = oacc[b][4 * j + e] * inv;
                // values d = 32 b + 8 j + 4 half + e: chunk 4 b + j, half h
                const int pc = (4 * b + j) ^ oswz(col);
                *reinterpret_cast<bf16x4 *>(tile + col * ROWB + pc * 16 + half * 8) =
                    __builtin_convertvector(t, bf16x4);
            }
        // this wave's LDS writes complete before it reads other lanes' data
        asm volatile("" ::: "memory");
        __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0)
        asm volatile("" ::: "memory");
        __bf16 *obase = reinterpret_cast<__bf16 *>(a.o);
#pragma unroll
        for (int k = 0; k < 32 * CHK / 64; ++k) {
            const int rr = lane / CHK + k * (64 / CHK);
            const int c = lane % CHK;
            const u32x4 val =
                *reinterpret_cast<const u32x4 *>(tile + rr * ROWB + ((c ^ oswz(rr)) << 4));
            if (row_base + rr < r1)
                *reinterpret_cast<u32x4 *>(
                    obase + ((seq_off + row_base + rr) * a.hq + head) * (int64_t)D + c * 8) = val;
        }
        if (a.lse && half == 0 && row_valid)
            a.lse[(int64_t)head * a.total_tokens + seq_off + my_row] = row_lse;
        return;
    }
    if (!row_valid)
        return;

    if (part_base >= 0) {
        const int64_t prow = (int64_t)(part_base + (my_row - r0)) * a.hq + head;
        float *po = a.part_o + prow * D;
#pragma unroll
        for (int b = 0; b < D_BLOCKS; ++b)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                f32x4 t;
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    t[e] = oacc[b][4 * j + e] * inv;
                *reinterpret_cast<f32x4 *>(po + b * 32 + 8 * j + 4 * half) = t;
            }
        if (half == 0)
            a.part_lse[prow] = row_lse;
        return;
    }

    const int64_t orow = ((seq_off + my_row) * a.hq + head) * (int64_t)D;
    if (a.o_f32) {
        float *op = reinterpret_cast<float *>(a.o) + orow;
#pragma unroll
        for (int b = 0; b < D_BLOCKS; ++b)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                f32x4 t;
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    t[e] = oacc[b][4 * j + e] * inv;
                *reinterpret_cast<f32x4 *>(op + b * 32 + 8 * j + 4 * half) = t;
            }
    } else {
        __bf16 *op = reinterpret_cast<__bf16 *>(a.o) + orow;
#pragma unroll
        for (int b = 0; b < D_BLOCKS; ++b)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                f32x4 t;
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    t[e] = oacc[b][4 * j + e] * inv;
                *reinterpret_cast<bf16x4 *>(op + b * 32 + 8 * j + 4 * half) =
                    __builtin_convertvector(t, bf16x4);
            }
    }
    if (a.lse && half == 0)
        a.lse[(int64_t)head * a.total_tokens + seq_off + my_row] = row_lse;
}

// Multi-unit form of the tile kernel for workgroups of five to eight waves
// (Q tiles in their own LDS region) over streaming and causal items.  A work
// unit is one (item, row block) of the schedule for one kv head; workgroup w
// owns kv head w % hkv and the units slot, slot + n_slots, slot + 2 n_slots,
// ... (slot = w / hkv, at most upw of them), so the units in flight on the
// chip at any time are neighbouring q-tiles of each kv head and share their
// band K/V tiles in L2.  The units of a workgroup run as one continuous
// pipeline of 64-key steps: the copies of K(j+1) and V(j) cross from one
// unit into the next, each wave copies the next unit's Q rows into its LDS Q
// tile while the current unit runs and reads them just before the next
// unit's first matrix phase, and the finished unit's epilogue (normalise,
// stage the bf16 rows in the now free Q tile, store whole rows) runs in the
// softmax phase of the next unit's first step.  The per-unit costs of a
// workgroup launch (schedule read, Q and first K tile from HBM, pipeline
// fill and drain, the gap before the next workgroup) are paid once per
// workgroup instead of once per unit.
//
// Before the pipeline starts, the workgroup turns its items into two LDS
// tables: one record per unit (rows, sequence, output slot, first step) and
// one word per pipeline step: the absolute token of the step's first key
// (bits 6 and up; trimmed steps never start past their sequence) and the
// number of its 64 keys that lie in the sequence, minus one (bits 0-5).  The
// step loop then carries only the step index, the current unit's index, its
// rows and the first step of the next unit.
constexpr int kMaxUnits = 128;    // units per workgroup
constexpr int kMaxSteps = 4096;   // pipeline steps per workgroup
constexpr int64_t kMaxUnitsTokens = int64_t(1) << 26;  // tokens a step word can hold
constexpr int kUnitWords = 12;    // unit record (see UnitField)
enum UnitField {
    U_START = 0, U_N, U_SEQ_OFF, U_SEQ_LEN, U_WR0, U_R1, U_PART, U_STREAM, U_A_LO, U_NA,
    U_B_LO, U_PART_ROW0
};

template <int D, int NW>
__global__ __launch_bounds__(NW * 64, 1) void attn_units_kernel(FwdArgs a, int32_t kind)
{
    constexpr int ROW_BYTES = 2 * D;
    constexpr int CHUNKS = D / 8;
    constexpr int TILE_BYTES = kStep * ROW_BYTES;
    constexpr int STAGE_BYTES = 2 * TILE_BYTES;
    constexpr int N_STAGES = 2;
    constexpr int ROWS_PER_DMA = 1024 / ROW_BYTES;
    constexpr int N_DMA = kStep / ROWS_PER_DMA;
    constexpr int N_COPY_WAVES = NW - NW / 2;
    constexpr int COPIES = (N_DMA + N_COPY_WAVES - 1) / N_COPY_WAVES;
    constexpr int QK_STEPS = D / 16;
    constexpr int D_BLOCKS = D / 32;
    constexpr int MFMA_SLOTS = 2 * QK_STEPS + 4 * D_BLOCKS;
    constexpr int COPY_STRIDE = MFMA_SLOTS / (2 * COPIES) > 0
                                    ? MFMA_SLOTS / (2 * COPIES) : 1;
    constexpr int QTILE_BYTES = 32 * ROW_BYTES;
    constexpr int QREGION = N_STAGES * STAGE_BYTES;
    static_assert(NW * QTILE_BYTES > STAGE_BYTES, "Q tiles have their own region");
    __shared__ __attribute__((aligned(1024))) unsigned char smem[QREGION + NW * QTILE_BYTES];
    __shared__ int32_t itab[kMaxUnits * kItemWords];  // the units' schedule items
    // unit records, then one private slot per wave (units without steps)
    __shared__ int32_t utab[(kMaxUnits + NW) * kUnitWords];
    __shared__ int32_t stab[kMaxSteps];               // step words
    typedef __attribute__((address_space(3))) int32_t lds_i32;
    // Kernel arguments used only at unit boundaries (Q copies, epilogue),
    // and the records of the current and next units, are held one word per
    // lane in a vector register each and read with v_readlane where used:
    // they take no scalar registers across the step loop and no memory
    // round trip at a boundary.
    struct BoundaryArgs {
        const uint16_t *q;
        void *o;
        float *lse, *part_o, *part_lse;
        int64_t total_tokens;
        int32_t hq, o_f32;
    };
    constexpr int kArgWords = (int)(sizeof(BoundaryArgs) / 4);
    static_assert(kArgWords <= 64 && kUnitWords <= 64, "one word per lane");
    __shared__ BoundaryArgs bargs;

    const int32_t *sched = a.sched;
    const int g = blockIdx.x % a.hkv;
    const int slot = blockIdx.x / a.hkv;
    const int n_my = min(a.upw, (a.n_units - slot + a.n_slots - 1) / a.n_slots);
    if (slot >= a.n_slots || n_my <= 0)
        return;
    if (!header_ok(sched, a.total_tokens, a.n_items, kind) || a.list_words != 0 ||
        n_my > kMaxUnits) {
        poison_outputs(a.o, a.o_f32, a.lse, a.total_tokens, a.hq, D, blockIdx.x, gridDim.x);
        return;
    }
    for (int t = threadIdx.x; t < n_my * kItemWords; t += NW * 64) {
        const int u = slot + (t / kItemWords) * a.n_slots;
        const int item = u / a.subtiles;
        itab[t] = sched[kHdrWords + (int64_t)item * kItemWords + t % kItemWords];
    }
    if (threadIdx.x == 0)
        bargs = BoundaryArgs{a.q, a.o, a.lse, a.part_o, a.part_lse, a.total_tokens, a.hq,
                             a.o_f32};
    __syncthreads();

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int half = lane >> 5;
    const int col = lane & 31;
    // The lane index as the compiler cannot see it: per-lane addresses of the
    // rarely run unit-boundary code (Q copies, epilogue) are derived from it,
    // so they are recomputed there instead of being hoisted out of the step
    // loop into registers that would stay live across every step.
    auto opaque_lane = [&]() TA_INLINE -> int {
        int x = lane;
        asm volatile("" : "+v"(x));
        return x;
    };
    const int args_v = lane < kArgWords ? ((lds_i32 *)&bargs)[lane] : 0;
    auto args = [&]() TA_INLINE -> BoundaryArgs {
        int av = args_v;
        asm volatile("" : "+v"(av));  // read here, not hoisted into scalars
        uint32_t v[kArgWords];
#pragma unroll
        for (int i = 0; i < kArgWords; ++i)
            v[i] = (uint32_t)__builtin_amdgcn_readlane(av, i);
        return __builtin_bit_cast(BoundaryArgs, v);
    };
    const int waves_per_head = a.rows_per_wg / 32;
    const int head = g * a.group + wave / waves_per_head;
    const int wave_row = (wave % waves_per_head) * 32;  // first row of the wave in a unit
    const float c = a.scale_log2;
    const int tps = a.tile / kStep;
    // unit record k, one word per lane; field f of it
    auto rec_of = [&](int ku) TA_INLINE -> int {
        return lane < kUnitWords
                   ? ((lds_i32 *)utab)[__builtin_amdgcn_readfirstlane(ku) * kUnitWords + lane]
                   : 0;
    };
    auto fld = [](int rv, int f) TA_INLINE -> int { return __builtin_amdgcn_readlane(rv, f); };

    const uint32_t smem_addr =
        (uint32_t)(uintptr_t)(__attribute__((address_space(3))) void *)smem;
    const uint32_t qtile_lds = smem_addr + QREGION + wave * QTILE_BYTES;
    // Copy the wave's 32 Q rows of unit ku into its LDS Q tile (rows past the
    // unit's rows repeat its last row).
    auto copy_q = [&](int rv) TA_INLINE {
        const int r1 = fld(rv, U_R1);
        const int row_base = fld(rv, U_WR0) + wave_row;
        const int q_row0 = min(row_base, r1 - 1);
        const int q_tok = fld(rv, U_SEQ_OFF) + q_row0;
        const BoundaryArgs ka = args();
        const int hq = ka.hq;
        const uint16_t *qb = ka.q + ((int64_t)q_tok * hq + head) * (int64_t)D;
        const uint32_t q_pitch = (uint32_t)(hq * ROW_BYTES);
        const int ln = opaque_lane();
#pragma unroll
        for (int i = 0; i < QTILE_BYTES / 1024; ++i) {
            const int row = i * (1024 / ROW_BYTES) + ln / CHUNKS;
            const int rr = min(row_base + row, r1 - 1) - q_row0;
            const uint32_t off = __umul24((uint32_t)rr, q_pitch) +
                                 (uint32_t)(((ln % CHUNKS) ^ kswz<D>(row)) << 4);
            copy_to_lds16(qb, off, qtile_lds + i * 1024);
        }
    };
    bf16x8 qf[QK_STEPS];
    auto read_q = [&]() TA_INLINE {
        const int ln = opaque_lane();
        const int cl = ln & 31, hf = ln >> 5;
        const unsigned char *qt = smem + QREGION + wave * QTILE_BYTES + cl * ROW_BYTES;
#pragma unroll
        for (int s = 0; s < QK_STEPS; ++s)
            qf[s] = *reinterpret_cast<const bf16x8 *>(qt + (((2 * s + hf) ^ kswz<D>(cl)) << 4));
    };

    f32x16 oacc[D_BLOCKS];
#pragma unroll
    for (int b = 0; b < D_BLOCKS; ++b)
        oacc[b] = f32x16{};

    // Epilogue of unit ku: O (or its normalised fp32 partial) and LSE of the
    // wave's rows, from oacc and the unit's l / m.  bf16 rows are staged in
    // the wave's Q tile (free: the next unit's Q has been read) and stored
    // whole.  Addresses: a uniform base at the wave's first row plus a
    // 32-bit per-lane offset.
    auto epilogue = [&](int rv, float l_sum, float m_row) TA_INLINE {
        const int r1 = fld(rv, U_R1);
        const int row_base = fld(rv, U_WR0) + wave_row;
        if (row_base >= r1)
            return;  // a ragged unit: this wave has no rows
        // partial row of sequence row r: part + r (a unit without partials
        // has U_PART = -1)
        const bool has_part = fld(rv, U_PART) >= 0;
        const int part = has_part ? fld(rv, U_PART_ROW0) : 0;
        const int64_t row_tok = (int64_t)fld(rv, U_SEQ_OFF) + row_base;
        const int ln = opaque_lane();
        const int col = ln & 31, half = ln >> 5;
        const bool row_valid = row_base + col < r1;
        const float l_tot = pair_sum(l_sum);
        const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
        const float row_lse = l_tot > 0.f ? (m_row + __log2f(l_tot)) * kLn2 : -INFINITY;
        const BoundaryArgs ka = args();
        const int hq = ka.hq;
        const uint32_t hd = (uint32_t)(hq * D);  // elements per token
        float *lse_row = nullptr;
        if (has_part)
            lse_row = ka.part_lse + ((int64_t)(part + row_base) * hq + head);
        else if (ka.lse)
            lse_row = ka.lse + (int64_t)head * ka.total_tokens + row_tok;
        const uint32_t lse_step = has_part ? (uint32_t)hq : 1u;
        if (!has_part && !ka.o_f32) {
            constexpr int ROWB = D * 2;
            constexpr int CHK = ROWB / 16;
            static_assert(32 * ROWB == QTILE_BYTES, "an output tile fills a Q tile");
            unsigned char *tile = smem + QREGION + wave * QTILE_BYTES;
            auto oswz = [](int r) { return D == 128 ? (r & 15) : ((r >> 1) & 7); };
#pragma unroll
            for (int b = 0; b < D_BLOCKS; ++b)
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    f32x4 t;
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        t[e] = oacc[b][4 * j + e] * inv;
                    const int pc = (4 * b + j) ^ oswz(col);
                    *reinterpret_cast<bf16x4 *>(tile + col * ROWB + pc * 16 + half * 8) =
                        __builtin_convertvector(t, bf16x4);
                }
            asm volatile("" ::: "memory");
            __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0)
            asm volatile("" ::: "memory");
            char *obase = reinterpret_cast<char *>(
                reinterpret_cast<__bf16 *>(ka.o) + (row_tok * hq + head) * (int64_t)D);
            constexpr int NCH = 32 * CHK / 64;  // 16-byte pieces per lane
            u32x4 val[NCH];
#pragma unroll
            for (int kk = 0; kk < NCH; ++kk) {  // every LDS read first, then the stores
                const int rr = ln / CHK + kk * (64 / CHK);
                const int cc = ln % CHK;
                val[kk] = *reinterpret_cast<const u32x4 *>(tile + rr * ROWB +
                                                           ((cc ^ oswz(rr)) << 4));
            }
#pragma unroll
            for (int kk = 0; kk < NCH; ++kk) {
                const int rr = ln / CHK + kk * (64 / CHK);
                const int cc = ln % CHK;
                if (row_base + rr < r1)
                    *reinterpret_cast<u32x4 *>(obase + (uint64_t)((uint32_t)rr * hd * 2u +
                                                                  (uint32_t)cc * 16u)) = val[kk];
            }
            // the staged tile is read before the Q tile is reused
            asm volatile("" ::: "memory");
            __builtin_amdgcn_s_waitcnt(0xc07f);
            asm volatile("" ::: "memory");
        } else if (row_valid) {
            float *po = has_part
                            ? ka.part_o + ((int64_t)(part + row_base) * hq + head) * D
                            : reinterpret_cast<float *>(ka.o) + (row_tok * hq + head) * D;
            const uint32_t lane_off = (uint32_t)col * hd + 4u * (uint32_t)half;
#pragma unroll
            for (int b = 0; b < D_BLOCKS; ++b)
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    f32x4 t;
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        t[e] = oacc[b][4 * j + e] * inv;
                    *reinterpret_cast<f32x4 *>(po + (uint64_t)(lane_off + b * 32 + 8 * j)) = t;
                }
        }
        if (lse_row && half == 0 && row_valid)
            lse_row[(uint64_t)((uint32_t)col * lse_step)] = row_lse;
    };

    // Pass 1 (every wave, scalar): validate each item (a malformed one
    // poisons the outputs before any work), pick the workgroup's rows, trim
    // the key runs to them (as the single-unit kernel does) and append a
    // record for every unit with steps.  Units without rows here are
    // dropped; a unit with rows but no steps (an empty split of a Last
    // q-tile) is written at once (zero partials, LSE -inf).
    int n_run = 0, n_total = 0;
    for (int k = 0; k < n_my; ++k) {
        lds_i32 *w = (lds_i32 *)itab + k * kItemWords;
        const int seq_off = __builtin_amdgcn_readfirstlane(w[I_SEQ_OFF]);
        const int seq_len = __builtin_amdgcn_readfirstlane(w[I_SEQ_LEN]);
        const int r0 = __builtin_amdgcn_readfirstlane(w[I_R0]);
        const int r1 = __builtin_amdgcn_readfirstlane(w[I_R1]);
        const int ka0 = __builtin_amdgcn_readfirstlane(w[I_KA0]);
        const int ka1 = __builtin_amdgcn_readfirstlane(w[I_KA1]);
        const int kb0 = __builtin_amdgcn_readfirstlane(w[I_KB0]);
        const int kb1 = __builtin_amdgcn_readfirstlane(w[I_KB1]);
        const int mode = __builtin_amdgcn_readfirstlane(w[I_MODE]);
        const int part_base = __builtin_amdgcn_readfirstlane(w[I_PART_BASE]);
        if (seq_off < 0 || seq_len < 0 || (int64_t)seq_off + seq_len > a.total_tokens ||
            r0 < 0 || r1 > seq_len || r0 >= r1 || ka0 < 0 || ka1 < ka0 || kb0 < 0 ||
            kb1 < kb0 || (mode != kModeStreaming && mode != kModeCausal) ||
            (part_base >= 0 && part_base + (r1 - r0) > a.n_partial_rows)) {
            poison_outputs(a.o, a.o_f32, a.lse, a.total_tokens, a.hq, D, blockIdx.x,
                           gridDim.x);
            poison_item_rows(a.o, a.o_f32, a.lse, a.part_o, a.part_lse, a.total_tokens, a.hq,
                             D, a.n_partial_rows, a.tile, seq_off, r0, r1, part_base);
            return;
        }
        const int sub = (slot + k * a.n_slots) % a.subtiles;
        const int wr0 = r0 + sub * a.rows_per_wg;
        if (wr0 >= r1)
            continue;
        const bool stream = mode == kModeStreaming;
        int a_lo = ka0 * tps, a_hi = ka1 * tps, b_lo = kb0 * tps, b_hi = kb1 * tps;
        const int wr_last = min(wr0 + a.rows_per_wg, r1) - 1;
        trim_runs(stream, a.sink, a.window, wr0, wr_last, a_lo, a_hi, b_lo, b_hi);
        const int na = a_hi - a_lo;
        const int n = na + (b_hi - b_lo);
        const int rec[kUnitWords] = {n_total, n, seq_off, seq_len, wr0, r1, part_base,
                                     stream ? 1 : 0, a_lo, na, b_lo, part_base - r0};
        if (n > 0 && (n_total + n > kMaxSteps || n_run >= kMaxUnits)) {
            poison_outputs(a.o, a.o_f32, a.lse, a.total_tokens, a.hq, D, blockIdx.x,
                           gridDim.x);
            return;
        }
        // every wave writes the same record words (one word per lane); a
        // unit without steps goes to the wave's private slot, is written
        // through the epilogue (oacc is zero) and dropped
        const int rslot = n == 0 ? kMaxUnits + wave : n_run;
        if (lane < kUnitWords) {
            int v = rec[0];
#pragma unroll
            for (int f = 1; f < kUnitWords; ++f)
                v = lane == f ? rec[f] : v;
            utab[rslot * kUnitWords + lane] = v;
        }
        if (n == 0) {
            __builtin_amdgcn_s_waitcnt(0xc07f);
            epilogue(rec_of(rslot), 0.f, -INFINITY);
            continue;
        }
        ++n_run;
        n_total += n;
    }
    __syncthreads();  // unit records written (the same words by every wave)
    if (n_total == 0)
        return;
    // Pass 2: wave w fills the step records of units w, w + NW, ...
    for (int ku = wave; ku < n_run; ku += NW) {
        const int rv = rec_of(ku);
        const int start = fld(rv, U_START), n = fld(rv, U_N);
        const int seq_off = fld(rv, U_SEQ_OFF), key_max = fld(rv, U_SEQ_LEN) - 1;
        const int a_lo = fld(rv, U_A_LO), na = fld(rv, U_NA), b_lo = fld(rv, U_B_LO);
        for (int s = lane; s < n; s += 64) {
            const int key0 = s < na ? (a_lo + s) * kStep : (b_lo + (s - na)) * kStep;
            stab[start + s] = ((seq_off + key0) << 6) | min(key_max - key0, kStep - 1);
        }
    }
    __syncthreads();

    // K/V tile copies (as the single-unit kernel) from a step record: the
    // absolute token of the tile's first row and its valid rows - 1; rows
    // past the sequence end read its last row (they lie beyond every row of
    // the unit, so the causal mask removes them).
    const uint16_t *kbase = a.k + (int64_t)g * D;
    const uint16_t *vbase = a.v + (int64_t)g * D;
    const int tok_stride = a.hkv * D;
    const bool copy_wave = wave < N_COPY_WAVES;
    const int dma_row_in = lane / CHUNKS;
    const int dma_pc = lane % CHUNKS;
    const uint32_t kx0 = (uint32_t)((dma_pc ^ kswz<D>(dma_row_in)) << 4);
    const uint32_t vx0 = (uint32_t)((dma_pc ^ vswz<D>(dma_row_in)) << 4);
    const uint32_t row_stride_bytes = 2u * (uint32_t)tok_stride;
    const uint32_t dma_off0 =
        __umul24((uint32_t)(wave * ROWS_PER_DMA + dma_row_in), row_stride_bytes);
    const uint32_t dma_off_step = (uint32_t)(N_COPY_WAVES * ROWS_PER_DMA) * row_stride_bytes;
    constexpr bool XR_PER_WAVE = D == 128 ? N_COPY_WAVES % 4 == 0 : N_COPY_WAVES % 2 == 0;
    struct TileCopy {
        const uint16_t *base;
        uint32_t lds;
        uint32_t lim;
    };
    auto srec = [&](int j) TA_INLINE -> uint32_t {
        return (uint32_t)__builtin_amdgcn_readfirstlane(
            ((lds_i32 *)stab)[__builtin_amdgcn_readfirstlane(j)]);
    };
    auto plan_copy = [&](const uint16_t *src, uint32_t w, int buf, bool is_v) TA_INLINE -> TileCopy {
        w = (uint32_t)__builtin_amdgcn_readfirstlane(w);  // uniform (a step word)
        TileCopy t;
        t.base = src + (int64_t)(w >> 6) * tok_stride;
        t.lim = (w & (kStep - 1)) * row_stride_bytes;
        t.lds = smem_addr + buf * STAGE_BYTES + (is_v ? TILE_BYTES : 0) + wave * 1024;
        // opaque: each copy adds its own offset (one scalar add) instead of
        // every copy address of both stages being held in its own register
        asm volatile("" : "+s"(t.lds));
        return t;
    };
    auto issue_copy = [&](const TileCopy &t, int i, bool is_v) TA_INLINE {
        const int m = wave + i * N_COPY_WAVES;
        if constexpr (N_DMA % N_COPY_WAVES != 0) {
            if (m >= N_DMA)
                return;
        }
        const uint32_t xr = is_v ? vx0 : (kx0 ^ (uint32_t)(kswz<D>(m * ROWS_PER_DMA) << 4));
        uint32_t off;
        if constexpr (XR_PER_WAVE)
            off = min(dma_off0 + (uint32_t)i * dma_off_step + xr, t.lim + xr);
        else
            off = min(dma_off0 + (uint32_t)i * dma_off_step, t.lim) + xr;
        copy_to_lds16(t.base, off, t.lds + i * (N_COPY_WAVES * 1024));
    };
    TileCopy cp_k{}, cp_v{};
    auto issue_slot = [&](int cidx) TA_INLINE {
        if (cidx < COPIES)
            issue_copy(cp_k, cidx, false);
        else
            issue_copy(cp_v, cidx - COPIES, true);
    };
    auto copy_hook = [&](int mslot) TA_INLINE {
        if (mslot % COPY_STRIDE == COPY_STRIDE - 1 && mslot / COPY_STRIDE < 2 * COPIES)
            issue_slot(mslot / COPY_STRIDE);
    };
    auto no_hook = [](int) {};

    const int krow0 = perm_row(col);
    uint32_t koff[QK_STEPS];
#pragma unroll
    for (int s = 0; s < QK_STEPS; ++s)
        koff[s] = (uint32_t)(krow0 * ROW_BYTES + (((2 * s + half) ^ kswz<D>(krow0)) << 4));
    // (No K fragments are read ahead here, unlike the single-unit kernel:
    // the unit loop has no registers to spare for them.)
    constexpr int KPRE = 0;
    auto qk = [&](int buf, f32x16 (&sacc)[2], auto hook, auto pre, auto own) TA_INLINE {
        (void)pre;
        const unsigned char *kt = smem + buf * STAGE_BYTES;
        sacc[0] = f32x16{};
        sacc[1] = f32x16{};
#pragma unroll
        for (int s = 0; s < QK_STEPS; ++s) {
            const bf16x8 a0 = *reinterpret_cast<const bf16x8 *>(kt + koff[s]);
            const bf16x8 a1 =
                *reinterpret_cast<const bf16x8 *>(kt + koff[s] + 32 * ROW_BYTES);
            sacc[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, qf[s], sacc[0], 0, 0, 0);
            hook(2 * s);
            sacc[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, qf[s], sacc[1], 0, 0, 0);
            hook(2 * s + 1);
        }
        constexpr int n = 2 * QK_STEPS, ahead = 6;
        if constexpr (!decltype(own)::value) {
            // the caller schedules the reads of the whole phase
        } else {
            __builtin_amdgcn_sched_group_barrier(kSchedDsRead, ahead, 0);
#pragma unroll
            for (int i = 0; i < n - ahead; ++i) {
                __builtin_amdgcn_sched_group_barrier(kSchedMfma, 1, 0);
                __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 1, 0);
            }
            __builtin_amdgcn_sched_group_barrier(kSchedMfma, ahead, 0);
        }
    };
    const int vrow0 = 8 * half + ((lane & 15) >> 2);
    const int tr_d = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
    uint32_t voff[D_BLOCKS];
#pragma unroll
    for (int b = 0; b < D_BLOCKS; ++b) {
        const int d = 32 * b + tr_d;
        voff[b] = (uint32_t)(vrow0 * ROW_BYTES + (((d >> 3) ^ vswz<D>(vrow0)) << 4) +
                             (d & 7) * 2);
    }
    auto pv = [&](int buf, const bf16x8 (&pf)[2][2], auto hook, auto own) TA_INLINE {
        const unsigned char *vt = smem + buf * STAGE_BYTES + TILE_BYTES;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
            for (int s2 = 0; s2 < 2; ++s2)
#pragma unroll
                for (int b = 0; b < D_BLOCKS; ++b) {
                    s16x4 part[2];
#pragma unroll
                    for (int i2 = 0; i2 < 2; ++i2)
                        part[i2] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                            (lds_s16x4 *)(vt + voff[b] +
                                          (kb * 32 + s2 * 16 + 4 * i2) * ROW_BYTES));
                    const bf16x8 af = __builtin_bit_cast(
                        bf16x8, __builtin_shufflevector(part[0], part[1], 0, 1, 2, 3, 4, 5,
                                                        6, 7));
                    oacc[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af, pf[kb][s2],
                                                                     oacc[b], 0, 0, 0);
                    hook(2 * QK_STEPS + (kb * 2 + s2) * D_BLOCKS + b);
                }
        if constexpr (decltype(own)::value) {
            constexpr int n = 4 * D_BLOCKS, ahead = 4;
            __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 2 * ahead, 0);
#pragma unroll
            for (int i = 0; i < n - ahead; ++i) {
                __builtin_amdgcn_sched_group_barrier(kSchedMfma, 1, 0);
                __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 2, 0);
            }
            __builtin_amdgcn_sched_group_barrier(kSchedMfma, ahead, 0);
        }
    };
    // Reads of a whole matrix phase in one sequence (as in the single-unit
    // kernel): the reads of MFMA i + 6 are issued just before MFMA i.
    auto sched_phase = [&](auto pre) TA_INLINE {
        constexpr bool PRE = false;
        (void)pre;
        constexpr int NQ = 2 * QK_STEPS, N = NQ + 4 * D_BLOCKS, ahead = 6;
        constexpr int first = phase_reads<NQ, N, KPRE, PRE>(0, ahead);
        if constexpr (first > 0)
            __builtin_amdgcn_sched_group_barrier(kSchedDsRead, first, 0);
        static_for<0, N>([&](auto ic) TA_INLINE {
            constexpr int nr = phase_reads<NQ, N, KPRE, PRE>(decltype(ic)::value + ahead, 1);
            __builtin_amdgcn_sched_group_barrier(kSchedMfma, 1, 0);
            if constexpr (nr > 0)
                __builtin_amdgcn_sched_group_barrier(kSchedDsRead, nr, 0);
        });
    };

    // The current unit, as the mask needs it (uniform).
    int ku = 0;                        // current unit
    int next_start = 0;                // first step of unit ku + 1 (n_total: none)
    int cur_row_base = 0, cur_row_hi = 0, cur_stream = 0, cur_seq_off = 0;
    int rec_cur = rec_of(0);                           // current unit
    int rec_nxt = n_run > 1 ? rec_of(1) : rec_cur;     // the next one
    auto enter_unit = [&](int k) TA_INLINE {
        ku = k;
        next_start = k + 1 < n_run ? fld(rec_nxt, U_START) : n_total;
        cur_seq_off = fld(rec_cur, U_SEQ_OFF);
        const int r1 = fld(rec_cur, U_R1);
        cur_row_base = fld(rec_cur, U_WR0) + wave_row;
        cur_row_hi = min(r1 - 1, cur_row_base + 31);
        cur_stream = fld(rec_cur, U_STREAM);
    };

    // Masks of one step.  A step can cross the diagonal (causal test), the
    // window edge of streaming rows (window test, the sink excepted) or
    // both; each case gets its own branch-free selects.  The window tests
    // use the sign of a difference as the select mask (a vector operation
    // per element, no lane mask in scalar registers: batches of compares
    // into lane masks would take dozens of scalar registers).
    auto keep_if = [](float sc, int m) TA_INLINE -> float {
        // m = -1: keep the score, m = 0: -inf
        return __builtin_bit_cast(float, (__builtin_bit_cast(uint32_t, sc) & (uint32_t)m) |
                                              (0xff800000u & ~(uint32_t)m));
    };
    auto mask_step = [&](int key0, f32x16 (&sacc)[2]) TA_INLINE {
        const int my_row = cur_row_base + col;
        const bool need_causal = key0 + kStep - 1 > cur_row_base;
        const bool need_window = cur_stream && key0 + kStep - 1 >= a.sink &&
                                 cur_row_hi - key0 >= a.window;
        const int lim = my_row - key0 - 8 * half;  // key offset <= lim: causal
        if (!need_window) {
            if (need_causal) {
#pragma unroll
                for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                    for (int v = 0; v < 16; ++v) {
                        const int off = kb * 32 + key_of_reg(v, 0);
                        sacc[kb][v] = off <= lim ? sacc[kb][v] : -INFINITY;
                    }
            }
            return;
        }
        const int win_lim = lim - a.window;             // offset > win_lim: in the window
        const int sink_lim = a.sink - key0 - 8 * half;  // offset < sink_lim: a sink key
        if (key0 + kStep - 1 <= cur_row_base - a.window) {
            // before every row's window (and diagonal): only sink keys remain
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int off = kb * 32 + key_of_reg(v, 0);
                    sacc[kb][v] = keep_if(sacc[kb][v], (off - sink_lim) >> 31);
                }
            return;
        }
        if (!need_causal && key0 >= a.sink) {
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int off = kb * 32 + key_of_reg(v, 0);
                    sacc[kb][v] = keep_if(sacc[kb][v], (win_lim - off) >> 31);
                }
            return;
        }
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int off = kb * 32 + key_of_reg(v, 0);
                const int m = ~((lim - off) >> 31) & (((off - sink_lim) >> 31) | ((win_lim - off) >> 31));
                sacc[kb][v] = keep_if(sacc[kb][v], m);
            }
    };
    auto step_needs_mask = [&](int key0) TA_INLINE -> bool {
        return (key0 + kStep - 1 > cur_row_base) ||
               (cur_stream && key0 + kStep - 1 >= a.sink && cur_row_hi - key0 >= a.window);
    };

    float m_ref = -INFINITY;
    float m_cur = -INFINITY;  // as in the single-unit kernel
    float l_run = 0.f;
    bool fresh = true;  // the unit's first softmax: no reference maximum on any lane
    auto softmax = [&](f32x16 (&sacc)[2], bf16x8 (&pf)[2][2]) TA_INLINE {
        auto exp_step = [&](float m_use) TA_INLINE -> float {
            float psum = 0.f;
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int s2 = 0; s2 < 2; ++s2) {
                    f32x8 t;
#pragma unroll
                    for (int e = 0; e < 8; ++e) {
                        t[e] = __builtin_amdgcn_exp2f(
                            __builtin_fmaf(sacc[kb][8 * s2 + e], c, -m_use));
                        psum = (kb | s2 | e) ? psum + t[e] : t[e];  // exp2 is never -0
                    }
                    pf[kb][s2] = __builtin_convertvector(t, bf16x8);
                }
            return psum;
        };
        // The first step of a unit has no reference on any lane: it goes
        // straight to the re-base (its first pass would be discarded).
        float psum = INFINITY;
        if (!fresh)
            psum = exp_step(m_cur);
        fresh = false;
        const bool bad = !(psum <= kRescaleBound);
        if (__builtin_amdgcn_ballot_w64(bad) != 0) {
            float mx = -INFINITY;
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int v = 0; v < 16; ++v)
                    mx = fmaxf(mx, sacc[kb][v]);
            mx = pair_max(mx);
            const float m_new = fmaxf(m_ref, mx * c);
            const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
            const float alpha = __builtin_amdgcn_exp2f(m_ref - m_use);
            l_run *= alpha;
#pragma unroll
            for (int b = 0; b < D_BLOCKS; ++b)
                oacc[b] *= alpha;
            m_ref = m_new;
            m_cur = m_new;
            psum = exp_step(m_use);
        }
        l_run += psum;
    };

    // Step words, read one phase ahead of their use: wk and wv for the
    // copies of K(j+1) and V(j) in the matrix phase of step j (steps past the
    // last one copy a repeat of the last K tile into parts of the stage
    // nobody reads), wx for the mask of the next softmax phase.
    uint32_t wk = 0, wv = 0, wx = 0;
    auto plan_step_copies = [&](auto stage) TA_INLINE {
        const int nbuf = 1 - (int)stage;
        cp_k = plan_copy(kbase, wk, nbuf, false);
        cp_v = plan_copy(vbase, wv, nbuf, true);
    };

    const int n_group1 = NW / 2;
    const int group = wave >= NW - n_group1 ? 1 : 0;
    f32x16 s_acc[2];
    bf16x8 p_acc[2][2];
    // prep() runs inside the phase, so that its scalar work (planning the
    // phase's copies) can overlap the first LDS reads.
    auto no_prep = []() {};
    auto do_m = [&](auto stage, bool has_qk, bool has_pv, auto hook, auto pre,
                    auto prep) TA_INLINE {
        __builtin_amdgcn_sched_barrier(0);
        __builtin_amdgcn_s_setprio(1);
        __builtin_amdgcn_sched_barrier(0);
        prep();
        const int buf = stage;
        if (has_qk && has_pv) {
            qk(buf, s_acc, hook, pre, std::false_type{});
            pv(buf, p_acc, hook, std::false_type{});
            sched_phase(pre);
        } else {
            if (has_qk)
                qk(buf, s_acc, hook, pre, std::true_type{});
            if (has_pv)
                pv(buf, p_acc, hook, std::true_type{});
        }
        __builtin_amdgcn_sched_barrier(0);
        __builtin_amdgcn_s_setprio(0);
        __builtin_amdgcn_sched_barrier(0);
    };
    auto do_x = [&]() TA_INLINE {
        const int key0 = (int)(__builtin_amdgcn_readfirstlane(wx) >> 6) - cur_seq_off;
        if (step_needs_mask(key0))
            mask_step(key0, s_acc);
        softmax(s_acc, p_acc);
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
            for (int s2 = 0; s2 < 2; ++s2)
                fence_regs(p_acc[kb][s2]);
        fence_regs(l_run);
        fence_regs(m_ref);
        fence_regs(m_cur);
    };
    auto end_phase = [&](bool wait_copies) TA_INLINE {
        __builtin_amdgcn_sched_barrier(0);
        if (wait_copies)
            wait_vmcnt(0);
        barrier_no_fence();
        __builtin_amdgcn_sched_barrier(0);
    };
    // Unit boundary, in the softmax phase of the new unit's first step
    // (after the matrix phase that finished the old unit's PV): write the old
    // unit, make the new one current, start copying the Q rows of the one
    // after it.
    auto boundary = [&]() TA_INLINE {
        epilogue(rec_cur, l_run, m_ref);
#pragma unroll
        for (int b = 0; b < D_BLOCKS; ++b)
            oacc[b] = f32x16{};
        m_ref = -INFINITY;
        m_cur = -INFINITY;
        l_run = 0.f;
        fresh = true;
        rec_cur = rec_nxt;
        rec_nxt = ku + 2 < n_run ? rec_of(ku + 2) : rec_cur;
        enter_unit(ku + 1);
        if (ku + 1 < n_run)
            copy_q(rec_nxt);
    };
    using Stage0 = std::integral_constant<int, 0>;
    using Stage1 = std::integral_constant<int, 1>;

    // Prologue: every wave copies its Q rows of the first unit, the copy
    // waves copy K(0) into stage 0; after the barrier each wave reads its Q
    // and starts copying the next unit's Q rows.
    enter_unit(0);
    copy_q(rec_cur);
    if (copy_wave) {
        cp_k = plan_copy(kbase, srec(0), 0, false);
#pragma unroll
        for (int cidx = 0; cidx < COPIES; ++cidx)
            issue_slot(cidx);
    }
    end_phase(true);
    read_q();
    __builtin_amdgcn_s_waitcnt(0xc07f);  // Q read before its tile is refilled
    if (n_run > 1)
        copy_q(rec_nxt);
    if (group == 0) {
        wk = srec(min(1, n_total - 1));
        wv = srec(0);
        do_m(Stage0{}, true, false, copy_hook, std::false_type{},
             [&]() TA_INLINE { plan_step_copies(Stage0{}); });
#pragma unroll
        for (int cidx = 0; cidx < 2 * COPIES; ++cidx)
            if (cidx * COPY_STRIDE + COPY_STRIDE - 1 >= 2 * QK_STEPS)
                issue_slot(cidx);
        end_phase(false);
        // softmax of step j (its word is wv), then the words of step j + 1
        auto x_phase = [&](int j) TA_INLINE {
            const int nv = ((lds_i32 *)stab)[min(j + 1, n_total - 1)];
            const int nk = ((lds_i32 *)stab)[min(j + 2, n_total - 1)];
            wx = wv;
            do_x();
            wv = (uint32_t)__builtin_amdgcn_readfirstlane(nv);
            wk = (uint32_t)__builtin_amdgcn_readfirstlane(nk);
        };
        x_phase(0);
        end_phase(true);
        // the Q copy of the next unit has landed at every unit start: the
        // last phase of each step waits for this wave's copies
        auto step = [&](int j, auto stage) TA_INLINE {
            const bool bnd = j == next_start;
            if (bnd)
                read_q();
            do_m(stage, true, true, copy_hook, std::false_type{},
                 [&]() TA_INLINE { plan_step_copies(stage); });
            end_phase(false);
            if (bnd)
                boundary();
            x_phase(j);
            end_phase(true);
        };
        int j = 1;
        for (; j + 1 < n_total; j += 2) {
            step(j, Stage1{});
            step(j + 1, Stage0{});
        }
        if (j < n_total)
            step(j++, Stage1{});
        do_m(j & 1, false, true, no_hook, std::false_type{}, no_prep);
        end_phase(false);
        end_phase(false);
    } else {
        end_phase(false);
        int nx = ((lds_i32 *)stab)[0];
        do_m(Stage0{}, true, false, no_hook, std::false_type{}, no_prep);
        end_phase(false);
        // the word of step j - 1 was read during the matrix phase before
        auto step = [&](int j, auto stage) TA_INLINE {
            if (j - 1 == next_start)
                boundary();
            wx = (uint32_t)__builtin_amdgcn_readfirstlane(nx);
            do_x();
            end_phase(false);
            if (j == next_start) {
                wait_vmcnt(0);  // the next unit's Q rows have landed
                read_q();
            }
            nx = ((lds_i32 *)stab)[j];
            do_m(stage, true, true, no_hook, std::false_type{}, no_prep);
            end_phase(false);
        };
        int j = 1;
        for (; j + 1 < n_total; j += 2) {
            step(j, Stage1{});
            step(j + 1, Stage0{});
        }
        if (j < n_total)
            step(j++, Stage1{});
        if (j - 1 == next_start)
            boundary();
        wx = (uint32_t)__builtin_amdgcn_readfirstlane(nx);
        do_x();
        end_phase(false);
        do_m(j & 1, false, true, no_hook, std::false_type{}, no_prep);
        end_phase(false);
    }
    epilogue(rec_cur, l_run, m_ref);
}

// LSE-weighted merge of the split partials of one q-tile (the Last rows of
// Triangle attention, or a block-sparse q-tile cut into chunks).  One wave
// per (row, query head) of merge item x: the wave reduces max and sum of the
// split LSEs across its lanes, then accumulates the weighted partial rows.
template <int D>
__device__ __forceinline__ bool merge_item_ok(const MergeArgs &a, const int32_t *x)
{
    const int64_t seq_off = x[M_SEQ_OFF];
    const int32_t r0 = x[M_R0], r1 = x[M_R1], ns = x[M_SPLITS], pb = x[M_PART_BASE];
    const int rows = r1 - r0;
    return rows >= 1 && rows <= a.tile && ns >= 1 && pb >= 0 &&
           pb + (int64_t)ns * rows <= a.n_partial_rows && seq_off >= 0 && r0 >= 0 &&
           seq_off + r1 <= a.total_tokens;
}

template <int D>
__device__ __forceinline__ void merge_row(const MergeArgs &a, const int32_t *x, int rank,
                                          int head, int lane)
{
    const int64_t seq_off = x[M_SEQ_OFF];
    const int32_t r0 = x[M_R0], r1 = x[M_R1], ns = x[M_SPLITS], pb = x[M_PART_BASE];
    const int rows = r1 - r0;
    if (rank >= rows)
        return;
    const int row = r0 + rank;

    auto lse_of = [&](int c) -> float {
        return a.part_lse[((int64_t)pb + (int64_t)c * rows + rank) * a.hq + head];
    };
    float mx = -INFINITY;
    for (int c = lane; c < ns; c += 64)
        mx = fmaxf(mx, lse_of(c));
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1)
        mx = fmaxf(mx, __shfl_xor(mx, off));
    const float m_use = (mx == -INFINITY) ? 0.f : mx;
    float den = 0.f;
    for (int c = lane; c < ns; c += 64)
        den += __expf(lse_of(c) - m_use);
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1)
        den += __shfl_xor(den, off);

    constexpr int PER = D / 64;  // elements per lane
    float acc[PER];
#pragma unroll
    for (int e = 0; e < PER; ++e)
        acc[e] = 0.f;
    // Partial rows of consecutive splits lie rows * hq * D floats apart.  The
    // loads of UNROLL splits (indices clamped to the last split) are issued
    // before any is used, so the wave keeps that many rows in flight; only
    // the splits that exist are added, in split order.
    const int64_t split_stride = (int64_t)rows * a.hq * D;
    const float *po0 = a.part_o + (((int64_t)pb + rank) * a.hq + head) * D + PER * lane;
    constexpr int UNROLL = 8;
    for (int c = 0; c < ns; c += UNROLL) {
        float t[UNROLL][PER], l[UNROLL];
#pragma unroll
        for (int u = 0; u < UNROLL; ++u) {
            const int cu = min(c + u, ns - 1);
            const float *po = po0 + (int64_t)cu * split_stride;
            if constexpr (PER == 2) {
                const f32x2 v = *reinterpret_cast<const f32x2 *>(po);
                t[u][0] = v[0];
                t[u][PER - 1] = v[1];
            } else {
                t[u][0] = po[0];
            }
            l[u] = lse_of(cu);
        }
#pragma unroll
        for (int u = 0; u < UNROLL; ++u) {
            if (c + u < ns) {
                const float wgt = __expf(l[u] - m_use);
#pragma unroll
                for (int e = 0; e < PER; ++e)
                    acc[e] += wgt * t[u][e];
            }
        }
    }
    const float inv = den > 0.f ? 1.f / den : 0.f;
    const int64_t orow = ((seq_off + row) * a.hq + head) * (int64_t)D;
    if (a.o_f32) {
        float *op = reinterpret_cast<float *>(a.o) + orow;
        if constexpr (PER == 2) {
            f32x2 t = {acc[0] * inv, acc[PER - 1] * inv};
            *reinterpret_cast<f32x2 *>(op + 2 * lane) = t;
        } else {
            op[lane] = acc[0] * inv;
        }
    } else {
        __bf16 *op = reinterpret_cast<__bf16 *>(a.o) + orow;
        if constexpr (PER == 2) {
            f32x2 t = {acc[0] * inv, acc[PER - 1] * inv};
            *reinterpret_cast<bf16x2 *>(op + 2 * lane) = __builtin_convertvector(t, bf16x2);
        } else {
            op[lane] = (__bf16)(acc[0] * inv);
        }
    }
    if (a.lse && lane == 0)
        a.lse[(int64_t)head * a.total_tokens + seq_off + row] =
            den > 0.f ? m_use + __logf(den) : -INFINITY;
}

// Grid: x covers the tile * hq (row, head) waves of one merge item, four per
// workgroup; y strides over the merge items.
template <int D>
__global__ __launch_bounds__(256) void merge_kernel(MergeArgs a)
{
    const int32_t *sched = a.sched;
    const int64_t block = (int64_t)blockIdx.y * gridDim.x + blockIdx.x;
    const int64_t n_blocks = (int64_t)gridDim.x * gridDim.y;
    if (!header_ok(sched, a.total_tokens, a.n_items, a.kind) || sched[H_TILE] != a.tile) {
        poison_outputs(a.o, a.o_f32, a.lse, a.total_tokens, a.hq, D, block, n_blocks);
        return;
    }
    const int32_t *mi = sched + kHdrWords + (int64_t)a.n_items * kItemWords;
    for (int m = blockIdx.y; m < a.n_merges; m += gridDim.y)
        if (!merge_item_ok<D>(a, mi + (int64_t)m * kMergeWords)) {
            poison_outputs(a.o, a.o_f32, a.lse, a.total_tokens, a.hq, D, block, n_blocks);
            return;
        }
    const int lane = threadIdx.x & 63;
    const int w = (int)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (w >= a.tile * a.hq)
        return;
    const int head = w % a.hq;
    const int rank = w / a.hq;  // row within the merge item
    for (int m = blockIdx.y; m < a.n_merges; m += gridDim.y)
        merge_row<D>(a, mi + (int64_t)m * kMergeWords, rank, head, lane);
}

// Rows per workgroup: the largest of 128, 64, 32 that divides the tile and
// keeps G * R / 32 <= 8 waves.
int rows_per_wg(int group, int tile)
{
    for (int r = 128; r >= 32; r /= 2)
        if (r <= tile && group * r / 32 <= 8)
            return r;
    return 32;
}

template <int D, bool LIST>
hipError_t launch_tile_as(int nw, dim3 grid, const FwdArgs &a, int kind, hipStream_t s)
{
    switch (nw) {
    case 2: hipLaunchKernelGGL((attn_tile_kernel<D, 2, false, LIST>), grid, dim3(128), 0, s, a, kind); break;
    case 4: hipLaunchKernelGGL((attn_tile_kernel<D, 4, false, LIST>), grid, dim3(256), 0, s, a, kind); break;
    case 5: hipLaunchKernelGGL((attn_tile_kernel<D, 5, false, LIST>), grid, dim3(320), 0, s, a, kind); break;
    case 6: hipLaunchKernelGGL((attn_tile_kernel<D, 6, false, LIST>), grid, dim3(384), 0, s, a, kind); break;
    // seven compute waves and a copier wave
    case 7: hipLaunchKernelGGL((attn_tile_kernel<D, 8, true, LIST>), grid, dim3(512), 0, s, a, kind); break;
    case 8: hipLaunchKernelGGL((attn_tile_kernel<D, 8, false, LIST>), grid, dim3(512), 0, s, a, kind); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

// Block-sparse schedules (list items) run the list form of the kernel.
template <int D>
hipError_t launch_tile(int nw, dim3 grid, const FwdArgs &a, int kind, hipStream_t s)
{
    return kind == TA_KIND_BLOCKSPARSE ? launch_tile_as<D, true>(nw, grid, a, kind, s)
                                       : launch_tile_as<D, false>(nw, grid, a, kind, s);
}

ta_status check_common(const char *fn, int want_kind, const void *q, const void *k,
                       const void *v, void *o, int32_t o_dtype,
                       const int32_t *sched_dev, const ta_schedule_info *info,
                       int64_t total_tokens, int32_t hq, int32_t hkv,
                       int32_t head_dim, float scale)
{
    if (!info)
        return fail(TA_ERR_INVALID_ARG, "%s: info is NULL", fn);
    if (info->version != TA_SCHEDULE_VERSION)
        return fail(TA_ERR_SCHEDULE_MISMATCH, "%s: schedule version %d != %d", fn,
                    info->version, TA_SCHEDULE_VERSION);
    if (info->kind != want_kind)
        return fail(TA_ERR_SCHEDULE_MISMATCH, "%s: schedule kind %d, need %d", fn,
                    info->kind, want_kind);
    if (total_tokens < 0)
        return fail(TA_ERR_INVALID_ARG, "%s: total_tokens < 0", fn);
    if (info->total_tokens != total_tokens)
        return fail(TA_ERR_SCHEDULE_MISMATCH,
                    "%s: schedule built for %lld tokens, call has %lld", fn,
                    (long long)info->total_tokens, (long long)total_tokens);
    if (hq <= 0 || hkv <= 0)
        return fail(TA_ERR_INVALID_ARG, "%s: hq and hkv must be positive", fn);
    if (hq % hkv != 0)
        return fail(TA_ERR_INVALID_ARG, "%s: hq %d not a multiple of hkv %d", fn, hq, hkv);
    if (hq / hkv > 8)
        return fail(TA_ERR_UNSUPPORTED, "%s: GQA group %d > 8", fn, hq / hkv);
    if (head_dim != 64 && head_dim != 128)
        return fail(TA_ERR_UNSUPPORTED, "%s: head_dim %d not in {64, 128}", fn, head_dim);
    if (info->tile != 64 && info->tile != 128)
        return fail(TA_ERR_UNSUPPORTED, "%s: tile %d not in {64, 128}", fn, info->tile);
    if (o_dtype != TA_OUT_BF16 && o_dtype != TA_OUT_F32)
        return fail(TA_ERR_INVALID_ARG, "%s: bad o_dtype %d", fn, o_dtype);
    if (!std::isfinite(scale) || !(scale > 0.f))
        return fail(TA_ERR_INVALID_ARG, "%s: softmax_scale must be finite and > 0", fn);
    if (info->n_items < 0 || info->n_merge_items < 0 || info->n_partial_rows < 0 ||
        info->n_last_rows < 0)
        return fail(TA_ERR_SCHEDULE_MISMATCH, "%s: corrupt schedule info", fn);
    {
        // words = header + items + merges (+ the k-tile lists of a block-sparse
        // schedule, whose length the window field records)
        const int64_t base = kHdrWords + (int64_t)info->n_items * kItemWords +
                             (int64_t)info->n_merge_items * kMergeWords;
        const int64_t lists = want_kind == TA_KIND_BLOCKSPARSE ? info->window : 0;
        if (lists < 0 || info->words != base + lists)
            return fail(TA_ERR_SCHEDULE_MISMATCH, "%s: schedule words %lld do not match "
                        "its items", fn, (long long)info->words);
    }
    if (total_tokens > 0 || info->n_items > 0) {
        if (!q || !k || !v || !o || !sched_dev)
            return fail(TA_ERR_INVALID_ARG, "%s: NULL q, k, v, o or schedule", fn);
        if (((uintptr_t)q | (uintptr_t)k | (uintptr_t)v | (uintptr_t)o) & 15)
            return fail(TA_ERR_INVALID_ARG, "%s: q, k, v and o must be 16-byte aligned", fn);
    }
    const int64_t subtiles = info->tile / rows_per_wg(hq / hkv, info->tile);
    if ((int64_t)info->n_items * subtiles * hkv > INT32_MAX)
        return fail(TA_ERR_UNSUPPORTED, "%s: grid too large", fn);
    // per-lane copy offsets use 24-bit multiplies of the K/V and Q row
    // pitches (2 hkv d and 2 hq d bytes; hq >= hkv)
    if (2LL * hq * head_dim >= (1LL << 24))
        return fail(TA_ERR_UNSUPPORTED, "%s: hq * head_dim too large", fn);
    return TA_OK;
}

FwdArgs make_args(const void *q, const void *k, const void *v, void *o,
                  int32_t o_dtype, float *lse, const int32_t *sched_dev,
                  const ta_schedule_info *info, int64_t total_tokens, int32_t hq,
                  int32_t hkv, float scale, float *part_o, float *part_lse)
{
    const int group = hq / hkv;
    const int R = rows_per_wg(group, info->tile);
    FwdArgs a;
    a.q = static_cast<const uint16_t *>(q);
    a.k = static_cast<const uint16_t *>(k);
    a.v = static_cast<const uint16_t *>(v);
    a.o = o;
    a.lse = lse;
    a.sched = sched_dev;
    a.part_o = part_o;
    a.part_lse = part_lse;
    a.total_tokens = total_tokens;
    a.hq = hq;
    a.hkv = hkv;
    a.group = group;
    a.n_items = info->n_items;
    a.n_partial_rows = info->n_partial_rows;
    a.list_base = kHdrWords + (int64_t)info->n_items * kItemWords +
                  (int64_t)info->n_merge_items * kMergeWords;
    a.list_words = info->words - a.list_base;
    a.sink = info->sink;
    a.window = info->window;
    a.tile = info->tile;
    a.rows_per_wg = R;
    a.subtiles = info->tile / R;
    a.o_f32 = o_dtype == TA_OUT_F32;
    a.scale_log2 = scale * kLog2e;
    a.n_units = 0;
    a.n_slots = 0;
    a.upw = 1;
    // Triangle schedules interleave their Last split items into the launch
    // (the slot arithmetic is 32-bit unsigned: (n_items + 1) n_lead < 2^32)
    const bool lead_fits = (uint64_t)(info->n_items + 1) * (uint64_t)info->n_last_items <
                           ((uint64_t)1 << 32);
    a.n_lead = info->kind == TA_KIND_TRIANGLE && lead_fits ? info->n_last_items : 0;
    return a;
}

template <int D>
hipError_t launch_units(int nw, dim3 grid, const FwdArgs &a, int kind, hipStream_t s)
{
    switch (nw) {
    case 5: hipLaunchKernelGGL((attn_units_kernel<D, 5>), grid, dim3(320), 0, s, a, kind); break;
    case 6: hipLaunchKernelGGL((attn_units_kernel<D, 6>), grid, dim3(384), 0, s, a, kind); break;
    case 7: hipLaunchKernelGGL((attn_units_kernel<D, 7>), grid, dim3(448), 0, s, a, kind); break;
    case 8: hipLaunchKernelGGL((attn_units_kernel<D, 8>), grid, dim3(512), 0, s, a, kind); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

// Units per workgroup of the multi-unit kernel for a Triangle pass, or 1
// for the single-unit kernel.  A unit boundary costs about as much as the
// per-workgroup costs it removes (measured: about 10 K cycles, the
// epilogue's normalisation, staging and stores beside the other group's
// MFMAs), the single-unit kernel reads K ahead where the multi-unit kernel
// has no registers to, and the pass runs at a power-limited clock, so the
// multi-unit kernel pays off only for short units, and less at d = 128 than
// at d = 64: on the paper's sink 8 / window 512 shape (10-12 steps) it is
// 4.6 % faster at d = 64 and about 1 % slower at d = 128 (four runs, each
// within about 1 % noise); at d = 128 units of 4-8 steps come out even and
// 36-step units at window 2048 6-10 % slower.  For units of at most
// short_unit_steps(d) steps: one workgroup per CU (256 CUs over the kv
// heads) when its units' steps fit the LDS step table, otherwise the fewest
// rounds of such workgroups whose units fit.  The environment variable
// TRIATTN_UNITS_PER_WG, read at every launch, overrides the count (1: the
// single-unit kernel) within the table limits: for tests and tuning.
int64_t short_unit_steps(int head_dim)
{
    return head_dim == 128 ? 8 : 16;
}
int units_per_wg(const FwdArgs &a, int kind, int nw, int64_t units, int32_t max_item_tiles,
                 int head_dim)
{
    if (kind != TA_KIND_TRIANGLE || nw < 5 || units > INT32_MAX ||
        a.total_tokens >= kMaxUnitsTokens || max_item_tiles < 1)
        return 1;
    const int64_t unit_steps = (int64_t)max_item_tiles * (a.tile / kStep);
    const int64_t cap = std::min<int64_t>(kMaxUnits, kMaxSteps / unit_steps);
    if (const char *env = std::getenv("TRIATTN_UNITS_PER_WG")) {
        const long forced = std::strtol(env, nullptr, 10);
        if (forced >= 1)
            return (int)std::max<int64_t>(1, std::min<int64_t>(forced, cap));
    }
    if (cap < 2 || unit_steps > short_unit_steps(head_dim))
        return 1;
    const int64_t slots = std::max<int64_t>(1, 256 / a.hkv);
    for (int64_t rounds = 1;; ++rounds) {
        const int64_t upw = (units + slots * rounds - 1) / (slots * rounds);
        if (upw <= cap)
            return (int)upw;
    }
}

ta_status launch_tiles(int kind, const FwdArgs &a_in, int32_t head_dim, int32_t max_item_tiles,
                       hipStream_t stream)
{
    if (a_in.n_items <= 0)
        return TA_OK;
    FwdArgs a = a_in;
    const int nw = a.group * a.rows_per_wg / 32;
    const int64_t units = (int64_t)a.n_items * a.subtiles;
    hipError_t err;
    // Triangle passes over workgroups of five to eight waves run several
    // units per workgroup (multi-unit kernel); the others one.
    const int upw = units_per_wg(a, kind, nw, units, max_item_tiles, head_dim);
    if (upw > 1) {
        a.n_units = (int32_t)units;
        a.upw = upw;
        a.n_slots = (int32_t)((units + upw - 1) / upw);
        dim3 grid((unsigned)((int64_t)a.n_slots * a.hkv));
        err = head_dim == 128 ? launch_units<128>(nw, grid, a, kind, stream)
                              : launch_units<64>(nw, grid, a, kind, stream);
    } else {
        dim3 grid((unsigned)(units * a.hkv));
        err = head_dim == 128 ? launch_tile<128>(nw, grid, a, kind, stream)
                              : launch_tile<64>(nw, grid, a, kind, stream);
    }
    if (err != hipSuccess)
        return fail(TA_ERR_HIP, "attention tile kernel launch failed: %s",
                    hipGetErrorString(err));
    return TA_OK;
}

ta_status launch_merge(void *o, int32_t o_dtype, float *lse, const int32_t *sched_dev,
                       const ta_schedule_info *info, int64_t total_tokens, int32_t hq,
                       int32_t head_dim, const float *part_o, const float *part_lse,
                       hipStream_t stream)
{
    // merge items come from Triangle (Last rows) or block-sparse schedules
    if (info->n_merge_items <= 0 || info->n_last_rows <= 0)
        return TA_OK;
    MergeArgs m;
    m.sched = sched_dev;
    m.part_o = part_o;
    m.part_lse = part_lse;
    m.o = o;
    m.lse = lse;
    m.total_tokens = total_tokens;
    m.hq = hq;
    m.n_items = info->n_items;
    m.n_merges = info->n_merge_items;
    m.n_partial_rows = info->n_partial_rows;
    m.n_last_rows = info->n_last_rows;
    m.o_f32 = o_dtype == TA_OUT_F32;
    m.kind = info->kind;
    m.tile = info->tile;
    dim3 grid((unsigned)((info->tile * hq + 3) / 4),
              (unsigned)std::min<int32_t>(info->n_merge_items, 65535));
    if (head_dim == 128)
        hipLaunchKernelGGL(merge_kernel<128>, grid, dim3(256), 0, stream, m);
    else
        hipLaunchKernelGGL(merge_kernel<64>, grid, dim3(256), 0, stream, m);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess)
        return fail(TA_ERR_HIP, "merge kernel launch failed: %s", hipGetErrorString(err));
    return TA_OK;
}

// Split the caller's workspace into the partial outputs and their LSE.
ta_status resolve_workspace(const char *fn, const ta_schedule_info *info, int32_t hq,
                            int32_t head_dim, const void *workspace,
                            size_t workspace_bytes, float **part_o, float **part_lse)
{
    *part_o = nullptr;
    *part_lse = nullptr;
    const size_t need = ta_workspace_bytes(info, hq, head_dim);
    if (need == 0)
        return TA_OK;
    if (!workspace || workspace_bytes < need)
        return fail(TA_ERR_WORKSPACE, "%s: workspace of %zu bytes needed, got %zu%s", fn,
                    need, workspace_bytes, workspace ? "" : " (NULL)");
    if ((uintptr_t)workspace & 15)
        return fail(TA_ERR_INVALID_ARG, "%s: workspace must be 16-byte aligned", fn);
    const size_t rows = (size_t)info->n_partial_rows * (size_t)hq;
    const size_t o_bytes = (rows * (size_t)head_dim * 4 + 255) & ~(size_t)255;
    *part_o = static_cast<float *>(const_cast<void *>(workspace));
    *part_lse = reinterpret_cast<float *>(static_cast<char *>(const_cast<void *>(workspace)) +
                                          o_bytes);
    return TA_OK;
}

}  // namespace
}  // namespace triattn

using namespace triattn;

extern "C" ta_status triangle_attn_tiles(const void *q, const void *k, const void *v,
                                         void *o, int32_t o_dtype, float *lse,
                                         const int32_t *sched_dev,
                                         const ta_schedule_info *info,
                                         int64_t total_tokens, int32_t hq, int32_t hkv,
                                         int32_t head_dim, float softmax_scale,
                                         void *workspace, size_t workspace_bytes,
                                         void *stream)
{
    clear_error();
    ta_status st = check_common("triangle_attn_tiles", TA_KIND_TRIANGLE, q, k, v, o,
                                o_dtype, sched_dev, info, total_tokens, hq, hkv,
                                head_dim, softmax_scale);
    if (st != TA_OK)
        return st;
    float *part_o, *part_lse;
    st = resolve_workspace("triangle_attn_tiles", info, hq, head_dim, workspace,
                           workspace_bytes, &part_o, &part_lse);
    if (st != TA_OK)
        return st;
    const FwdArgs a = make_args(q, k, v, o, o_dtype, lse, sched_dev, info, total_tokens,
                                hq, hkv, softmax_scale, part_o, part_lse);
    return launch_tiles(TA_KIND_TRIANGLE, a, head_dim, info->max_item_tiles,
                        static_cast<hipStream_t>(stream));
}

extern "C" ta_status triangle_attn_merge(void *o, int32_t o_dtype, float *lse,
                                         const int32_t *sched_dev,
                                         const ta_schedule_info *info,
                                         int64_t total_tokens, int32_t hq,
                                         int32_t head_dim, const void *workspace,
                                         size_t workspace_bytes, void *stream)
{
    clear_error();
    static const char fn[] = "triangle_attn_merge";
    if (!info)
        return fail(TA_ERR_INVALID_ARG, "%s: info is NULL", fn);
    if (info->version != TA_SCHEDULE_VERSION || info->kind != TA_KIND_TRIANGLE)
        return fail(TA_ERR_SCHEDULE_MISMATCH, "%s: need a Triangle schedule (version %d)",
                    fn, TA_SCHEDULE_VERSION);
    if (info->total_tokens != total_tokens)
        return fail(TA_ERR_SCHEDULE_MISMATCH,
                    "%s: schedule built for %lld tokens, call has %lld", fn,
                    (long long)info->total_tokens, (long long)total_tokens);
    if (hq <= 0)
        return fail(TA_ERR_INVALID_ARG, "%s: hq must be positive", fn);
    if (head_dim != 64 && head_dim != 128)
        return fail(TA_ERR_UNSUPPORTED, "%s: head_dim %d not in {64, 128}", fn, head_dim);
    if (o_dtype != TA_OUT_BF16 && o_dtype != TA_OUT_F32)
        return fail(TA_ERR_INVALID_ARG, "%s: bad o_dtype %d", fn, o_dtype);
    if (info->n_merge_items > 0 && (!o || !sched_dev))
        return fail(TA_ERR_INVALID_ARG, "%s: NULL o or schedule", fn);
    if ((uintptr_t)o & 15)
        return fail(TA_ERR_INVALID_ARG, "%s: o must be 16-byte aligned", fn);
    float *part_o, *part_lse;
    ta_status st = resolve_workspace(fn, info, hq, head_dim, workspace, workspace_bytes,
                                     &part_o, &part_lse);
    if (st != TA_OK)
        return st;
    return launch_merge(o, o_dtype, lse, sched_dev, info, total_tokens, hq, head_dim,
                        part_o, part_lse, static_cast<hipStream_t>(stream));
}

namespace {
// The two launches of a pass with split q-tiles (Triangle: Last rows;
// block-sparse: q-tiles with several items): tiles, then merge.
ta_status split_pass_fwd(const char *fn, int kind, const void *q, const void *k,
                         const void *v, void *o, int32_t o_dtype, float *lse,
                         const int32_t *sched_dev, const ta_schedule_info *info,
                         int64_t total_tokens, int32_t hq, int32_t hkv, int32_t head_dim,
                         float softmax_scale, void *workspace, size_t workspace_bytes,
                         void *stream)
{
    clear_error();
    ta_status st = check_common(fn, kind, q, k, v, o, o_dtype, sched_dev, info,
                                total_tokens, hq, hkv, head_dim, softmax_scale);
    if (st != TA_OK)
        return st;
    float *part_o, *part_lse;
    st = resolve_workspace(fn, info, hq, head_dim, workspace, workspace_bytes, &part_o,
                           &part_lse);
    if (st != TA_OK)
        return st;
    const hipStream_t s = static_cast<hipStream_t>(stream);
    const FwdArgs a = make_args(q, k, v, o, o_dtype, lse, sched_dev, info, total_tokens,
                                hq, hkv, softmax_scale, part_o, part_lse);
    st = launch_tiles(kind, a, head_dim, info->max_item_tiles, s);
    if (st != TA_OK)
        return st;
    return launch_merge(o, o_dtype, lse, sched_dev, info, total_tokens, hq, head_dim,
                        part_o, part_lse, s);
}
}  // namespace

extern "C" ta_status triangle_attn_fwd(const void *q, const void *k, const void *v,
                                       void *o, int32_t o_dtype, float *lse,
                                       const int32_t *sched_dev,
                                       const ta_schedule_info *info,
                                       int64_t total_tokens, int32_t hq, int32_t hkv,
                                       int32_t head_dim, float softmax_scale,
                                       void *workspace, size_t workspace_bytes,
                                       void *stream)
{
    return split_pass_fwd("triangle_attn_fwd", TA_KIND_TRIANGLE, q, k, v, o, o_dtype, lse,
                          sched_dev, info, total_tokens, hq, hkv, head_dim, softmax_scale,
                          workspace, workspace_bytes, stream);
}

namespace {
constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_dev[kMaxScratchDevices] = {};

// Device address of `scratch` on the stream's GPU, looked up once per GPU
// (with that GPU current) and kept.
ta_status scratch_address(const char *fn, hipStream_t stream, void **out)
{
    int dev = -1;
    hipError_t err = stream ? hipStreamGetDevice(stream, &dev) : hipGetDevice(&dev);
    if (err != hipSuccess)
        return fail(TA_ERR_HIP, "%s: no device for the stream: %s", fn,
                    hipGetErrorString(err));
    if (dev < 0 || dev >= kMaxScratchDevices)
        return fail(TA_ERR_UNSUPPORTED, "%s: device %d beyond %d", fn, dev,
                    kMaxScratchDevices);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_dev[dev]) {
        int cur = -1;
        err = hipGetDevice(&cur);
        if (err == hipSuccess && cur != dev)
            err = hipSetDevice(dev);
        void *p = nullptr;
        if (err == hipSuccess)
            err = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (cur >= 0 && cur != dev) {
            const hipError_t e2 = hipSetDevice(cur);
            if (err == hipSuccess)
                err = e2;
        }
        if (err != hipSuccess || !p)
            return fail(TA_ERR_HIP, "%s: scratch address on device %d: %s", fn, dev,
                        hipGetErrorString(err));
        g_scratch_dev[dev] = p;
    }
    *out = g_scratch_dev[dev];
    return TA_OK;
}
}  // namespace

extern "C" ta_status triangle_attn_fwd_noalloc(const void *q, const void *k, const void *v,
                                               void *o, int32_t o_dtype, float *lse,
                                               const int32_t *sched_dev,
                                               const ta_schedule_info *info,
                                               int64_t total_tokens, int32_t hq,
                                               int32_t hkv, int32_t head_dim,
                                               float softmax_scale, void *stream)
{
    static const char fn[] = "triangle_attn_fwd_noalloc";
    clear_error();
    ta_status st = check_common(fn, TA_KIND_TRIANGLE, q, k, v, o, o_dtype, sched_dev,
                                info, total_tokens, hq, hkv, head_dim, softmax_scale);
    if (st != TA_OK)
        return st;
    const size_t need = ta_workspace_bytes(info, hq, head_dim);
    if (need > (size_t)TA_NOALLOC_SCRATCH_BYTES)
        return fail(TA_ERR_WORKSPACE,
                    "%s: the split partials need %zu bytes, the library scratch holds "
                    "%zu: build the schedule with fewer splits or use triangle_attn_fwd",
                    fn, need, (size_t)TA_NOALLOC_SCRATCH_BYTES);
    void *ws = nullptr;
    if (need > 0) {
        st = scratch_address(fn, static_cast<hipStream_t>(stream), &ws);
        if (st != TA_OK)
            return st;
    }
    return split_pass_fwd(fn, TA_KIND_TRIANGLE, q, k, v, o, o_dtype, lse, sched_dev, info,
                          total_tokens, hq, hkv, head_dim, softmax_scale, ws,
                          ws ? (size_t)TA_NOALLOC_SCRATCH_BYTES : 0, stream);
}

extern "C" ta_status blocksparse_attn_fwd(const void *q, const void *k, const void *v,
                                          void *o, int32_t o_dtype, float *lse,
                                          const int32_t *sched_dev,
                                          const ta_schedule_info *info,
                                          int64_t total_tokens, int32_t hq, int32_t hkv,
                                          int32_t head_dim, float softmax_scale,
                                          void *workspace, size_t workspace_bytes,
                                          void *stream)
{
    return split_pass_fwd("blocksparse_attn_fwd", TA_KIND_BLOCKSPARSE, q, k, v, o, o_dtype,
                          lse, sched_dev, info, total_tokens, hq, hkv, head_dim,
                          softmax_scale, workspace, workspace_bytes, stream);
}

extern "C" ta_status causal_attn_fwd(const void *q, const void *k, const void *v,
                                     void *o, int32_t o_dtype, float *lse,
                                     const int32_t *sched_dev,
                                     const ta_schedule_info *info, int64_t total_tokens,
                                     int32_t hq, int32_t hkv, int32_t head_dim,
                                     float softmax_scale, void *stream)
{
    clear_error();
    ta_status st = check_common("causal_attn_fwd", TA_KIND_CAUSAL, q, k, v, o, o_dtype,
                                sched_dev, info, total_tokens, hq, hkv, head_dim,
                                softmax_scale);
    if (st != TA_OK)
        return st;
    const FwdArgs a = make_args(q, k, v, o, o_dtype, lse, sched_dev, info, total_tokens,
                                hq, hkv, softmax_scale, nullptr, nullptr);
    return launch_tiles(TA_KIND_CAUSAL, a, head_dim, info->max_item_tiles,
                        static_cast<hipStream_t>(stream));
}
