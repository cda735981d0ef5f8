// Region-contribution probe of libtriattn.so for gfx950 (MI355X).
//
// Sec. 2.2 measures how much a model output y depends on a section of the
// attention matrix with a probing variable theta that scales the attention
// probabilities elementwise (A_theta = theta (.) A, O = A_theta V).  At
// theta = 1 the derivative is d y / d theta_ij = A_ij <dO_i, V_j>, with dO the
// upstream gradient of the attention output, and Grad(M-hat, l) is its mean
// over the pairs of the section M-hat.  This file sums the derivative per
// query head over the three sections of Appendix A.3 (streaming, middle,
// last), which partition the causal mask; Sec. 3 ranks layers by the middle
// section's value to choose the Triangle layers.
//
// Probe kernel: a workgroup owns one kv head g, one block of R rows of each
// q-tile for each of the G query heads of g (so every K/V tile staged in
// LDS serves the whole GQA group) and one slot: an equal share of the kept
// k-tiles of the causal schedule's work items (a q-tile and its k-tiles up
// to the diagonal), the items laid end to end in schedule order.  A share
// is a run of chunks (an item's k-tiles from s0 to s1), so a q-tile's
// k-tiles may be spread over two or more workgroups: the probe's sums are
// additive over key ranges, and equal shares keep the pass from waiting on
// the longest q-tile (at 2K tokens one item per workgroup leaves the
// diagonal's last q-tile with 16 k-tiles against a mean of 8.5).  Each wave
// owns 32 rows of one head.  Per 64-key step it runs
// two bf16 MFMA 32x32x16 contractions with the same operand layout, S^T =
// K Q^T and dP^T = V dO^T (keys on the MFMA rows, queries on the columns), so
// a lane holds matching entries of both: it forms A = 2^(S c - lse log2 e)
// (c = scale log2 e; the row's LSE is an input, so no softmax state is
// carried) and adds A dP to the accumulator of the pair's section.  Per-step
// fp32 sums go into fp64 lane accumulators; each wave reduces them and writes
// one fp64 partial per (slot, 32-row block, head, section).  The reduce kernel sums
// the partials of each (head, section) in a fixed order, so results are
// deterministic.  Roofline: MFMA, 4 T^2 d flops per kept (q-tile, k-tile)
// pair and head, as the forward pass.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstdlib>
#include <numeric>
#include <type_traits>
#include <vector>

#include "triattn_device.h"
#include "triattn_internal.h"

namespace triattn {
namespace {

constexpr int kProbeStep = 64;  // keys per step
constexpr float kProbeLog2e = 1.4426950408889634f;
constexpr int kProbeCUs = 256;       // compute units of the MI355X
constexpr int kProbeMaxSlots = 512;  // workgroups per (kv head, row block), at most
// Cost of moving to the next item within a share, in 64-key steps: the
// pipeline drains, and the new q-tile's Q, dO and LSE rows arrive before
// its first matrix phase.  At 2K tokens charges of 3, 4 and 5 steps time the
// same and 2 is 12 % slower; 4 is the middle of that range.
constexpr int kProbeItemChange = 4;

struct ProbeArgs {
    const uint16_t *q;
    const uint16_t *k;
    const uint16_t *v;
    const uint16_t *dout;
    const float *lse;     // [hq, total] natural log
    const int32_t *sched;
    double *part;         // [n_slots * tile / 32, hq, 3]
    int64_t total_tokens;
    int32_t hq, hkv, group;
    int32_t n_items;
    int32_t tile;
    int32_t rows_per_wg;  // R
    int32_t subtiles;     // tile / R
    int32_t sink, window, last;
    float scale_log2;     // softmax scale * log2(e)
    int32_t n_slots;      // workgroups per (kv head, row block)
    int32_t per_item;     // 1: workgroup slot runs item slot whole
    int64_t total_cost;   // kept k-tiles per head (the items' costs summed)
};

// 16-byte chunk swizzle of LDS row r: the 32 rows one operand fetch reads
// land on distinct banks.
template <int D>
__device__ __forceinline__ int probe_swz(int r)
{
    return D == 128 ? (r & 15) : ((r >> 1) & 7);
}

// The tests combine with & (no short-circuit), so every header word is
// loaded before any test: one memory round trip instead of one per test.
__device__ __forceinline__ bool probe_header_ok(const int32_t *s, int64_t total,
                                                int32_t n_items, int32_t tile, int64_t kept)
{
    const int64_t t = (int64_t)(uint32_t)s[H_TOTAL_LO] | ((int64_t)s[H_TOTAL_HI] << 32);
    return (s[H_MAGIC] == TA_SCHEDULE_MAGIC) & (s[H_VERSION] == TA_SCHEDULE_VERSION) &
           (s[H_KIND] == TA_KIND_CAUSAL) & (s[H_TILE] == tile) & (t == total) &
           (s[H_ITEMS] == n_items) & (s[H_KEPT_TILES] == kept);
}

template <int D, int NW>
__global__ __launch_bounds__(NW * 64, NW == 4 ? 2 : 1) void probe_kernel(ProbeArgs a)
{
    constexpr int ROW_BYTES = 2 * D;
    constexpr int CHUNKS = D / 8;                       // 16-byte chunks per row
    constexpr int TILE_BYTES = kProbeStep * ROW_BYTES;  // one K or V tile
    constexpr int STAGE_BYTES = 2 * TILE_BYTES;         // K tile, then V tile
    constexpr int ROWS_PER_DMA = 1024 / ROW_BYTES;      // rows per wave copy
    constexpr int N_DMA = kProbeStep / ROWS_PER_DMA;    // wave copies per tile
    constexpr int N_COPY_WAVES = NW - NW / 2;           // the waves of group 0
    constexpr int COPIES = (N_DMA + N_COPY_WAVES - 1) / N_COPY_WAVES;  // per tile
    constexpr int QK = D / 16;                          // MFMA k-steps over d
    constexpr int MFMA_SLOTS = 4 * QK;                  // MFMAs of a matrix phase
    constexpr int COPY_STRIDE = MFMA_SLOTS / (2 * COPIES) > 0
                                    ? MFMA_SLOTS / (2 * COPIES) : 1;
    constexpr int NT = NW * 64;
    __shared__ __attribute__((aligned(1024))) uint8_t lds[2 * STAGE_BYTES];
    __shared__ int64_t wave_tot[NW];
    __shared__ int64_t first[4];  // first item of the share, lo, its prefix, hi

    const int per_slot = a.subtiles * a.hkv;
    const int slot = blockIdx.x / per_slot;
    const int rem = blockIdx.x - slot * per_slot;
    const int g = rem / a.subtiles;
    const int sub = rem - g * a.subtiles;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int h = lane >> 5;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wph = a.rows_per_wg / 32;  // waves per head
    const int head = g * a.group + wave / wph;
    const int rb = sub * wph + wave % wph;  // 32-row block within the q-tile
    // Ping-pong groups as in the forward tile kernel: waves w and w + 4
    // share a SIMD and sit in different groups; group 0 copies the K/V tiles.
    const int group = wave >= NW - NW / 2 ? 1 : 0;
    const bool copy_wave = wave < N_COPY_WAVES;

    const int32_t *sched = a.sched;
    // The item words are read without waiting for the header check, so that
    // both loads are in flight together (the host has checked that the
    // schedule holds n_items items, so the reads are in bounds either way).
    bool ok = probe_header_ok(sched, a.total_tokens, a.n_items, a.tile, a.total_cost);
    // The workgroup's share [lo, hi) of the kept 64-key steps (tile / 64 per
    // kept k-tile), counted over the items laid end to end in schedule order
    // from `pre` at item `item`: one whole item (per-item launch), or one of
    // n_slots shares of the total.  The shares are equal in a virtual cost
    // that charges each item kProbeItemChange steps on top of its own, placed
    // before its first step, so a share that walks many short items gets
    // fewer steps; a virtual position v inside item i (virtual prefix P) is
    // the real position P - i * kProbeItemChange + max(0, v - P -
    // kProbeItemChange).  At 2K tokens (16 items of 32, 30, .., 2 steps over
    // 16 slots) equal k-tile shares give one share 18 steps over three
    // items (four with equal step shares); virtual shares give the shares
    // that walk many short items fewer steps.
    const int spt = a.tile / kProbeStep;
    const int64_t total_steps = (int64_t)spt * a.total_cost;
    int item = 0;
    int64_t pre = 0, lo = 0, hi = 0;
    if (a.per_item) {
        item = slot;
        hi = (int64_t)spt * sched[kHdrWords + (int64_t)item * kItemWords + I_COST];
        ok = ok && hi >= 0;  // a negative cost would skip the item's checks
    } else {
        const int64_t vtotal = total_steps + (int64_t)kProbeItemChange * a.n_items;
        const int64_t per = (vtotal + a.n_slots - 1) / a.n_slots;
        const int64_t vlo = min((int64_t)slot * per, vtotal);
        const int64_t vhi = min(vlo + per, vtotal);
        lo = hi = pre = total_steps;  // an empty share is covered as it stands
        item = a.n_items;
        if (vlo < vhi) {
            // Items holding virtual positions vlo and vhi: thread t sums the
            // (virtual) costs of items
            // [t m, t m + m), a scan over the threads gives each its prefix,
            // and the threads whose items contain vlo and vhi record the
            // share's bounds.  The costs must add up to the header's total,
            // none negative.
            const int m = (a.n_items + NT - 1) / NT;
            const int i0 = min(tid * m, a.n_items), i1 = min(i0 + m, a.n_items);
            auto cost_of = [&](int i) -> int64_t {  // virtual, in steps
                return (int64_t)spt * sched[kHdrWords + (int64_t)i * kItemWords + I_COST] +
                       kProbeItemChange;
            };
            int64_t tsum = 0;
            bool neg = false;
            for (int i = i0; i < i1; ++i) {
                const int64_t c = cost_of(i);
                neg |= c < kProbeItemChange;  // a negative cost
                tsum += c;
            }
            int64_t x = tsum;  // inclusive scan over the wave
#pragma unroll
            for (int o = 1; o < 64; o <<= 1) {
                const int64_t y = __shfl_up(x, o);
                if (lane >= o)
                    x += y;
            }
            if (lane == 63)
                wave_tot[wave] = x;
            if (tid == 0) {
                first[0] = -1;
                first[3] = total_steps;  // vhi at the end of the last item
            }
            __syncthreads();
            int64_t p = x - tsum, total = 0;
            for (int w = 0; w < NW; ++w) {
                p += w < wave ? wave_tot[w] : 0;
                total += wave_tot[w];
            }
            for (int i = i0; i < i1; ++i) {
                const int64_t c = cost_of(i);
                const int64_t start = p - (int64_t)i * kProbeItemChange;  // real prefix
                if (p <= vlo && vlo < p + c) {
                    first[0] = i;
                    first[1] = start + max<int64_t>(0, vlo - p - kProbeItemChange);
                    first[2] = start;
                }
                if (p <= vhi && vhi < p + c)
                    first[3] = start + max<int64_t>(0, vhi - p - kProbeItemChange);
                p += c;
            }
            const bool any_neg = __syncthreads_or(neg);
            ok = ok && !any_neg && total == vtotal && first[0] >= 0;
            auto uniform = [](int64_t x) -> int64_t {
                const uint32_t l = __builtin_amdgcn_readfirstlane((uint32_t)x);
                const uint32_t h = __builtin_amdgcn_readfirstlane((uint32_t)(x >> 32));
                return (int64_t)(((uint64_t)h << 32) | l);
            };
            item = __builtin_amdgcn_readfirstlane((int)first[0]);
            lo = uniform(first[1]);
            pre = uniform(first[2]);
            hi = uniform(first[3]);
        }
    }

    const float c = a.scale_log2;
    const int tok_stride = a.hkv * D;
    const uint32_t row_stride_bytes = 2u * (uint32_t)tok_stride;  // < 2^24 (host check)
    const uint32_t smem_addr =
        (uint32_t)(uintptr_t)(__attribute__((address_space(3))) void *)lds;

    // A operand offsets: lane row r = lane % 32 of a 32-row half, chunk
    // (2 s + h) ^ swizzle(r); the second half (rows 32-63) adds 32 rows (its
    // swizzle is the same).
    const int r_lane = lane & 31;
    uint32_t aoff[QK];
#pragma unroll
    for (int s = 0; s < QK; ++s)
        aoff[s] = (uint32_t)(r_lane * ROW_BYTES + (((2 * s + h) ^ probe_swz<D>(r_lane)) << 4));

    // Copy m of a tile writes its rows m * ROWS_PER_DMA .. (1 KB): lane l
    // lands at row m * ROWS_PER_DMA + l / CHUNKS, stored chunk l % CHUNKS,
    // which holds logical chunk (l % CHUNKS) ^ swizzle(row); rows past the
    // last key of the sequence read that key (masked).  Group-0 wave w makes
    // copies m = w, w + N_COPY_WAVES, ... of each K and V tile.
    const int dma_row_in = lane / CHUNKS;
    const int dma_pc = lane % CHUNKS;
    struct TileCopy {
        const uint16_t *kb, *vb;  // row kc of K and V
        uint32_t lim;             // min(last key - kc, 63) * row pitch in bytes
        uint32_t lds;             // LDS address of the stage
    };
    TileCopy cp{};
    auto issue_copy = [&](int i, bool is_v) TA_INLINE {
        const int m = wave + i * N_COPY_WAVES;
        if constexpr (N_DMA % N_COPY_WAVES != 0) {
            if (m >= N_DMA)
                return;
        }
        const int row = m * ROWS_PER_DMA + dma_row_in;
        const uint32_t off = min(__umul24((uint32_t)row, row_stride_bytes), cp.lim) +
                             (uint32_t)((dma_pc ^ probe_swz<D>(row)) << 4);
        copy_to_lds16(is_v ? cp.vb : cp.kb, off,
                      cp.lds + (is_v ? TILE_BYTES : 0) + m * 1024);
    };
    auto issue_slot = [&](int cc) TA_INLINE {
        if (cc < COPIES)
            issue_copy(cc, false);
        else
            issue_copy(cc - COPIES, true);
    };
    auto copy_hook = [&](int slot_) TA_INLINE {
        if (slot_ % COPY_STRIDE == COPY_STRIDE - 1 && slot_ / COPY_STRIDE < 2 * COPIES)
            issue_slot(slot_ / COPY_STRIDE);
    };
    auto no_hook = [](int) {};
    // Burst form of the copies, for chunks whose K/V tiles all lie inside
    // the sequence (nothing to clamp): copy wave w copies the consecutive
    // 1 KB blocks w * COPIES .. w * COPIES + COPIES - 1 of a tile in one burst
    // with one M0 write, at the copy slots of the first K and the first V
    // copy; its lane offsets (row * pitch + swizzled chunk - i KB, i the
    // block's index in the burst, which the instruction offset adds back)
    // are constants of the lane.
    constexpr bool BURST = (COPIES == 2 || COPIES == 4) && N_DMA == COPIES * N_COPY_WAVES;
    constexpr int BURST_K_SLOT = COPY_STRIDE - 1;
    constexpr int BURST_V_SLOT = COPIES * COPY_STRIDE + COPY_STRIDE - 1;
    uint32_t boff[BURST ? COPIES : 1];
    if constexpr (BURST) {
#pragma unroll
        for (int i = 0; i < COPIES; ++i) {
            const int row = (wave * COPIES + i) * ROWS_PER_DMA + dma_row_in;
            boff[i] = __umul24((uint32_t)row, row_stride_bytes) - (uint32_t)(i * 1024) +
                      (uint32_t)((dma_pc ^ probe_swz<D>(row)) << 4);
        }
    }
    auto burst_hook = [&](int slot_) TA_INLINE {
        if constexpr (BURST) {
            const uint32_t blk = cp.lds + (uint32_t)(wave * COPIES * 1024);
            if (slot_ == BURST_K_SLOT)
                copy_burst_to_lds16<COPIES>(cp.kb, boff, blk);
            else if (slot_ == BURST_V_SLOT)
                copy_burst_to_lds16<COPIES>(cp.vb, boff, blk + TILE_BYTES);
        }
    };
    auto end_phase = [&](bool wait_copies) TA_INLINE {
        __builtin_amdgcn_sched_barrier(0);
        if (wait_copies)
            wait_vmcnt(0);
        barrier_no_fence();
        __builtin_amdgcn_sched_barrier(0);
    };
    using Stage0 = std::integral_constant<int, 0>;
    using Stage1 = std::integral_constant<int, 1>;

    double acc_s = 0.0, acc_m = 0.0, acc_l = 0.0;  // streaming / middle / last
    for (; ok && item < a.n_items && pre < hi; ++item) {
        const int32_t *it = sched + kHdrWords + (int64_t)item * kItemWords;
        const int64_t seq_off = it[I_SEQ_OFF];
        const int32_t seq_len = it[I_SEQ_LEN];
        const int32_t r0 = it[I_R0], r1 = it[I_R1];
        const int32_t ka0 = it[I_KA0], ka1 = it[I_KA1];
        const int64_t cost = it[I_COST];
        // guard against a malformed schedule: never touch memory outside it
        // (& without short-circuits: the item words are loaded together)
        ok = (it[I_MODE] == kModeCausal) & (it[I_KB0] == it[I_KB1]) & (seq_off >= 0) &
             (seq_len > 0) & (seq_off + seq_len <= a.total_tokens) & (r0 >= 0) & (r0 < r1) &
             (r1 <= seq_len) & (ka0 >= 0) & (ka1 >= ka0) & (cost == ka1 - ka0) &
             ((int64_t)ka1 * a.tile < (int64_t)seq_len + a.tile);
        if (!ok)
            break;
        const int s0 = (int)max<int64_t>(lo - pre, 0);  // the share's steps
        const int s1 = (int)min<int64_t>(hi - pre, spt * cost);  // of the item
        pre += spt * cost;
        const int wr0 = r0 + sub * a.rows_per_wg;  // first row of this workgroup
        if (wr0 >= r1)
            continue;  // ragged q-tile: no rows here (uniform)
        // keys past the workgroup's last row are masked for all its rows
        const int wg_last = min(wr0 + a.rows_per_wg, r1) - 1;
        const int key_begin = ka0 * a.tile + s0 * kProbeStep;
        const int key_end = min(ka0 * a.tile + s1 * kProbeStep, wg_last + 1);
        const int nsteps =
            key_end > key_begin ? (key_end - key_begin + kProbeStep - 1) / kProbeStep : 0;
        if (nsteps == 0)
            continue;  // the share holds no keys of these rows (uniform)

        const int row_base = wr0 + (wave % wph) * 32;
        const int my_row = row_base + r_lane;
        const bool row_valid = my_row < r1;
        const int load_row = row_valid ? my_row : r1 - 1;
        const int row_hi = min(row_base + 31, r1 - 1);  // last valid row of the wave
        const bool last_row = my_row >= seq_len - min(a.last, seq_len);
        const float lse2 = a.lse[(int64_t)head * a.total_tokens + seq_off + load_row] *
                           kProbeLog2e;

        // B operands: lane holds Q[row][16 s + 8 h ..] and dO[row][16 s + 8 h ..]
        bf16x8 qf[QK], df[QK];
        {
            const int64_t off = ((seq_off + load_row) * a.hq + head) * (int64_t)D + 8 * h;
#pragma unroll
            for (int s = 0; s < QK; ++s) {
                qf[s] = *reinterpret_cast<const bf16x8 *>(a.q + off + 16 * s);
                df[s] = *reinterpret_cast<const bf16x8 *>(a.dout + off + 16 * s);
            }
        }

        const int key_max = seq_len - 1;
        const uint16_t *kbase = a.k + (seq_off * a.hkv + g) * (int64_t)D;
        const uint16_t *vbase = a.v + (seq_off * a.hkv + g) * (int64_t)D;
        // K and V tiles of step j into LDS stage `buf`
        auto plan_copies = [&](int j, int buf) TA_INLINE {
            const int kc = min(key_begin + j * kProbeStep, key_max);
            cp.kb = kbase + (int64_t)kc * tok_stride;
            cp.vb = vbase + (int64_t)kc * tok_stride;
            cp.lim = (uint32_t)min(key_max - kc, kProbeStep - 1) * row_stride_bytes;
            cp.lds = smem_addr + buf * STAGE_BYTES;
        };

        f32x16 sacc[2], gacc[2];
        // Matrix phase of step j from LDS stage `stage`: S^T = K Q^T and
        // dP^T = V dO^T for the two 32-key halves, the four accumulator
        // chains interleaved so that dependent MFMAs do not stall.
        // The first KPRE operand fragments of a matrix phase (its first MFMAs'
        // K and V reads, in MFMA order) can be read ahead in the wave's vector
        // phase before it, when the stage has landed by then (group 1).
        constexpr int KPRE = 6;
        bf16x8 kpre[KPRE];
        auto frag = [&](const uint8_t *kt, int i) TA_INLINE -> bf16x8 {
            // read i of a matrix phase: s = i / 4; k0, v0, k1, v1
            const uint8_t *base = (i & 1) ? kt + TILE_BYTES : kt;
            return *reinterpret_cast<const bf16x8 *>(base + aoff[i / 4] +
                                                     ((i >> 1) & 1) * 32 * ROW_BYTES);
        };
        auto prefetch = [&](int buf) TA_INLINE {
            const uint8_t *kt = lds + buf * STAGE_BYTES;
#pragma unroll
            for (int i = 0; i < KPRE; ++i)
                kpre[i] = frag(kt, i);
        };
        // Matrix phase of step j from LDS stage `stage`: S^T = K Q^T and
        // dP^T = V dO^T for the two 32-key halves, the four accumulator
        // chains interleaved so that dependent MFMAs do not stall.  prep()
        // runs inside the phase, so that its scalar work (planning the
        // phase's copies) overlaps the first LDS reads.
        auto do_m = [&](auto stage, auto hook, auto pre, auto prep) TA_INLINE {
            constexpr bool PRE = decltype(pre)::value;
            __builtin_amdgcn_sched_barrier(0);
            __builtin_amdgcn_s_setprio(1);  // MFMA issue goes first on the SIMD
            __builtin_amdgcn_sched_barrier(0);
            prep();
            const uint8_t *kt = lds + (int)stage * STAGE_BYTES;
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) {
                sacc[kb] = f32x16{};
                gacc[kb] = f32x16{};
            }
#pragma unroll
            for (int s = 0; s < QK; ++s) {
                bf16x8 f[4];
#pragma unroll
                for (int u = 0; u < 4; ++u)
                    f[u] = (PRE && 4 * s + u < KPRE) ? kpre[4 * s + u] : frag(kt, 4 * s + u);
                sacc[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f[0], qf[s], sacc[0], 0, 0, 0);
                hook(4 * s);
                gacc[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f[1], df[s], gacc[0], 0, 0, 0);
                hook(4 * s + 1);
                sacc[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f[2], qf[s], sacc[1], 0, 0, 0);
                hook(4 * s + 2);
                gacc[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f[3], df[s], gacc[1], 0, 0, 0);
                hook(4 * s + 3);
            }
            constexpr int n = MFMA_SLOTS, ahead = 6;
            if constexpr (PRE) {
                // read r feeds MFMA KPRE + r: one read before each MFMA from
                // the first keeps them KPRE MFMAs ahead
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
            __builtin_amdgcn_sched_barrier(0);
            __builtin_amdgcn_s_setprio(0);
            __builtin_amdgcn_sched_barrier(0);
        };

        // Vector phase of step j: A dP per pair, summed per section.  Register
        // e of half kb holds key key0 + o(kb, e) + 4 h, o = 32 kb + (e & 3) +
        // 8 (e >> 2).  A step whose pairs are all of one section (streaming or
        // not) needs at most the causal test; only steps across a section
        // edge classify each pair.  Rows past the q-tile are dropped when the
        // chunk ends.
        double chunk_s = 0.0, chunk_o = 0.0;  // streaming / other (middle or last)
        auto do_x = [&](int j) TA_INLINE {
            const int key0 = key_begin + j * kProbeStep;
            const int lim = my_row - key0 - 4 * h;  // causal: o <= lim
            const bool causal_all = key0 + kProbeStep - 1 <= row_base;
            const bool strm_all = key0 + kProbeStep - 1 < a.sink || row_hi - key0 < a.window;
            const bool strm_none =
                key0 >= a.sink && row_base - (key0 + kProbeStep - 1) >= a.window;
            float ts = 0.f, to = 0.f;
            if (strm_all || strm_none) {
                float t = 0.f;
                if (causal_all) {
#pragma unroll
                    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                        for (int e = 0; e < 16; ++e)
                            t += __builtin_amdgcn_exp2f(fmaf(sacc[kb][e], c, -lse2)) *
                                 gacc[kb][e];
                } else {
#pragma unroll
                    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                        for (int e = 0; e < 16; ++e) {
                            const int o = 32 * kb + (e & 3) + 8 * (e >> 2);
                            const float pr =
                                __builtin_amdgcn_exp2f(fmaf(sacc[kb][e], c, -lse2)) *
                                gacc[kb][e];
                            t += o <= lim ? pr : 0.f;
                        }
                }
                ts = strm_all ? t : 0.f;
                to = strm_all ? 0.f : t;
            } else {
                const int slim = a.sink - key0 - 4 * h;  // sink key: o < slim
                const int wlim = lim - a.window;          // in the window: o > wlim
                float tv = 0.f;
#pragma unroll
                for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                    for (int e = 0; e < 16; ++e) {
                        const int o = 32 * kb + (e & 3) + 8 * (e >> 2);
                        const float pr =
                            __builtin_amdgcn_exp2f(fmaf(sacc[kb][e], c, -lse2)) * gacc[kb][e];
                        const float pv = o <= lim ? pr : 0.f;
                        tv += pv;
                        ts += ((o < slim) | (o > wlim)) ? pv : 0.f;
                    }
                to = tv - ts;
            }
            chunk_s += (double)ts;
            chunk_o += (double)to;
            fence_regs(chunk_s);
            fence_regs(chunk_o);
        };

        // Two-group ping-pong over the steps (the forward tile kernel's
        // schedule, with both operands of a step in one stage): group 0 runs
        // the matrix phase of step j in phase 2j and its vector phase in
        // phase 2j+1, group 1 one phase later.  Stage j & 1 holds K(j) and
        // V(j); during its matrix phase of step j group 0 copies K(j+1) and
        // V(j+1) into stage (j+1) & 1 (last read in phase 2j-1) and waits for
        // them at the end of phase 2j+1.  The last step's copies repeat its
        // own tiles into the other stage, which nobody reads.
        if (nsteps > 0) {
            if (copy_wave) {
                plan_copies(0, 0);
#pragma unroll
                for (int cc = 0; cc < 2 * COPIES; ++cc)
                    issue_slot(cc);
            }
            end_phase(true);  // K(0) and V(0) have landed
            if (group == 0) {
                auto run_group0 = [&](auto burst) TA_INLINE {
                    auto hook = [&](int slot_) TA_INLINE {
                        if constexpr (decltype(burst)::value)
                            burst_hook(slot_);
                        else
                            copy_hook(slot_);
                    };
                    auto step = [&](int j, auto stage) TA_INLINE {
                        do_m(stage, hook, std::false_type{}, [&]() TA_INLINE {
                            plan_copies(min(j + 1, nsteps - 1), 1 - (int)stage);
                        });
                        end_phase(false);
                        do_x(j);
                        end_phase(true);
                    };
                    int j = 0;
                    for (; j + 1 < nsteps; j += 2) {
                        step(j, Stage0{});
                        step(j + 1, Stage1{});
                    }
                    if (j < nsteps)
                        step(j, Stage0{});
                };
                // the chunk's steps are contiguous: every tile lies inside
                // the sequence when the last one does
                if constexpr (BURST) {
                    if (key_begin + nsteps * kProbeStep - 1 <= key_max)
                        run_group0(std::true_type{});
                    else
                        run_group0(std::false_type{});
                } else {
                    run_group0(std::false_type{});
                }
                end_phase(false);  // group 1's last vector phase
            } else {
                // group 1's matrix phase of step j reads stage j & 1, which
                // has landed before its vector phase of step j - 1: the
                // phase's first fragments are read at the start of that phase
                auto no_prep = []() {};
                prefetch(0);
                end_phase(false);  // group 0's first matrix phase
                do_m(Stage0{}, no_hook, std::true_type{}, no_prep);
                end_phase(false);
                auto step = [&](int j, auto stage) TA_INLINE {
                    prefetch(stage);
                    do_x(j - 1);
                    end_phase(false);
                    do_m(stage, no_hook, std::true_type{}, no_prep);
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
            }
        }
        if (row_valid) {
            acc_s += chunk_s;
            if (last_row)
                acc_l += chunk_o;
            else
                acc_m += chunk_o;
        }
    }
    ok = ok && pre >= hi;  // the items cover the share

#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
        acc_s += __shfl_xor(acc_s, off);
        acc_m += __shfl_xor(acc_m, off);
        acc_l += __shfl_xor(acc_l, off);
    }
    if (lane == 0) {
        // every partial is written (zero for an empty share), so the
        // workspace needs no clearing; a schedule that does not match the
        // call gives NaN sums
        double *pp = a.part + (((int64_t)slot * (a.tile / 32) + rb) * a.hq + head) * 3;
        const double bad = __builtin_nan("");
        pp[0] = ok ? acc_s : bad;
        pp[1] = ok ? acc_m : bad;
        pp[2] = ok ? acc_l : bad;
    }
}

// out[hr] = sum over blocks b of part[b, hr] (hr = head * 3 + section), in a
// fixed order: one wave per output, lane-strided sums, then an xor-shuffle
// tree.  Four outputs per workgroup.
__global__ __launch_bounds__(256) void probe_reduce_kernel(const double *part, int64_t n_blocks,
                                                           int32_t hq3, double *out)
{
    const int hr = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (hr >= hq3)
        return;
    const int lane = threadIdx.x & 63;
    double s = 0.0;
    for (int64_t b = lane; b < n_blocks; b += 64)
        s += part[b * hq3 + hr];
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1)
        s += __shfl_xor(s, off);
    if (lane == 0)
        out[hr] = s;
}

int probe_rows_per_wg(int group, int tile)
{
    for (int r = 128; r >= 32; r /= 2)
        if (r <= tile && group * r / 32 <= 8)
            return r;
    return 32;
}

// Work split of the probe over the workgroups of one (kv head, row block).
// Equal shares of the kept steps (with a charge per item change), one
// workgroup each, as many as fill every compute unit's resident workgroups
// once (two for workgroups of at most four waves, whose registers and LDS
// leave room for two per CU, else one), when the schedule's longest item is more than half a share: then one
// item per workgroup would leave the pass waiting on the longest q-tile (at
// 2K tokens: 16 k-tiles against a mean of 8.5).  Otherwise one workgroup per
// item, in schedule order (heaviest first): the workgroups running at a time
// then walk the same keys in step and share them in L2.  The environment
// variable TRIATTN_PROBE_SLOTS, read at every call, forces equal shares of
// that count (1 .. kProbeMaxSlots): for tests.
struct ProbeSplit {
    int64_t slots;
    bool per_item;
};
ProbeSplit probe_split(int nw, int64_t wgs_per_slot, const ta_schedule_info *info)
{
    if (const char *env = std::getenv("TRIATTN_PROBE_SLOTS")) {
        const long forced = std::strtol(env, nullptr, 10);
        if (forced >= 1)
            return {std::min<int64_t>(forced, kProbeMaxSlots), false};
    }
    const int64_t resident = (int64_t)kProbeCUs * (nw <= 4 ? 2 : 1);
    const int64_t slots =
        std::max<int64_t>(1, std::min<int64_t>(kProbeMaxSlots, resident / wgs_per_slot));
    if ((int64_t)info->max_item_tiles * slots * 2 <= info->kept_tiles_per_qhead)
        return {info->n_items, true};
    return {slots, false};
}

template <int D>
hipError_t launch_probe(int nw, dim3 grid, const ProbeArgs &a, hipStream_t s)
{
    switch (nw) {
    case 2: hipLaunchKernelGGL((probe_kernel<D, 2>), grid, dim3(128), 0, s, a); break;
    case 4: hipLaunchKernelGGL((probe_kernel<D, 4>), grid, dim3(256), 0, s, a); break;
    case 5: hipLaunchKernelGGL((probe_kernel<D, 5>), grid, dim3(320), 0, s, a); break;
    case 6: hipLaunchKernelGGL((probe_kernel<D, 6>), grid, dim3(384), 0, s, a); break;
    case 7: hipLaunchKernelGGL((probe_kernel<D, 7>), grid, dim3(448), 0, s, a); break;
    case 8: hipLaunchKernelGGL((probe_kernel<D, 8>), grid, dim3(512), 0, s, a); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace
}  // namespace triattn

using namespace triattn;

extern "C" size_t ta_probe_workspace_bytes(const ta_schedule_info *info, int32_t hq)
{
    if (!info || hq <= 0 || info->n_items <= 0 || info->tile < 32)
        return 0;
    // one partial per (workgroup slot, 32-row block, head, section)
    const size_t slots = (size_t)std::max<int64_t>(info->n_items, kProbeMaxSlots);
    return slots * (size_t)(info->tile / 32) * (size_t)hq * 3 * sizeof(double);
}

extern "C" ta_status region_grad_probe(const void *q, const void *k, const void *v,
                                       const void *dout, const float *lse,
                                       const int32_t *sched_dev, const ta_schedule_info *info,
                                       int64_t total_tokens, int32_t hq, int32_t hkv,
                                       int32_t head_dim, float softmax_scale, int32_t sink,
                                       int32_t window, int32_t last, double *region_sums,
                                       void *workspace, size_t workspace_bytes,
                                       void *stream_ptr)
{
    hipStream_t stream = static_cast<hipStream_t>(stream_ptr);
    clear_error();
    static const char fn[] = "region_grad_probe";
    if (!info)
        return fail(TA_ERR_INVALID_ARG, "%s: info is NULL", fn);
    if (info->version != TA_SCHEDULE_VERSION)
        return fail(TA_ERR_SCHEDULE_MISMATCH, "%s: schedule version %d != %d", fn,
                    info->version, TA_SCHEDULE_VERSION);
    if (info->kind != TA_KIND_CAUSAL)
        return fail(TA_ERR_SCHEDULE_MISMATCH, "%s: needs a causal schedule, got kind %d",
                    fn, info->kind);
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
    if (!std::isfinite(softmax_scale) || !(softmax_scale > 0.f))
        return fail(TA_ERR_INVALID_ARG, "%s: softmax_scale must be finite and > 0", fn);
    if (sink < 0 || window < 0 || last < 0)
        return fail(TA_ERR_INVALID_ARG, "%s: need sink, window, last >= 0", fn);
    if (info->n_items < 0 ||
        info->words != kHdrWords + (int64_t)info->n_items * kItemWords +
                           (int64_t)info->n_merge_items * kMergeWords)
        return fail(TA_ERR_SCHEDULE_MISMATCH, "%s: corrupt schedule info", fn);
    if (!region_sums || ((uintptr_t)region_sums & 7))
        return fail(TA_ERR_INVALID_ARG, "%s: region_sums must be a non-NULL 8-byte "
                    "aligned device array", fn);
    if (info->n_items > 0) {
        if (!q || !k || !v || !dout || !lse || !sched_dev)
            return fail(TA_ERR_INVALID_ARG, "%s: NULL q, k, v, dout, lse or schedule", fn);
        if (((uintptr_t)q | (uintptr_t)k | (uintptr_t)v | (uintptr_t)dout) & 15)
            return fail(TA_ERR_INVALID_ARG, "%s: q, k, v and dout must be 16-byte aligned", fn);
        if ((uintptr_t)lse & 3)
            return fail(TA_ERR_INVALID_ARG, "%s: lse must be 4-byte aligned", fn);
    }
    const size_t need = ta_probe_workspace_bytes(info, hq);
    if (need > 0 && (!workspace || workspace_bytes < need || ((uintptr_t)workspace & 7)))
        return fail(TA_ERR_WORKSPACE, "%s: workspace needs %zu bytes (8-byte aligned), "
                    "got %zu", fn, need, workspace_bytes);
    const int group = hq / hkv;
    const int R = probe_rows_per_wg(group, info->tile);
    const int64_t subtiles = info->tile / R;
    const int nw = group * R / 32;
    const ProbeSplit split = probe_split(nw, subtiles * hkv, info);
    const int64_t slots = split.slots;
    if (slots * subtiles * hkv > INT32_MAX)
        return fail(TA_ERR_UNSUPPORTED, "%s: grid too large", fn);
    // per-lane copy offsets use 24-bit multiplies of the K/V row pitch
    if (2LL * hkv * head_dim >= (1LL << 24))
        return fail(TA_ERR_UNSUPPORTED, "%s: hkv * head_dim too large", fn);

    double *part = static_cast<double *>(workspace);
    if (info->n_items > 0) {
        ProbeArgs a;
        a.q = static_cast<const uint16_t *>(q);
        a.k = static_cast<const uint16_t *>(k);
        a.v = static_cast<const uint16_t *>(v);
        a.dout = static_cast<const uint16_t *>(dout);
        a.lse = lse;
        a.sched = sched_dev;
        a.part = part;
        a.total_tokens = total_tokens;
        a.hq = hq;
        a.hkv = hkv;
        a.group = group;
        a.n_items = info->n_items;
        a.tile = info->tile;
        a.rows_per_wg = R;
        a.subtiles = (int32_t)subtiles;
        a.sink = sink;
        a.window = window;
        a.last = last;
        a.scale_log2 = softmax_scale * kProbeLog2e;
        a.n_slots = (int32_t)slots;
        a.per_item = split.per_item ? 1 : 0;
        a.total_cost = info->kept_tiles_per_qhead;
        dim3 grid((unsigned)(slots * subtiles * hkv));
        hipError_t err = head_dim == 128 ? launch_probe<128>(nw, grid, a, stream)
                                         : launch_probe<64>(nw, grid, a, stream);
        if (err != hipSuccess)
            return fail(TA_ERR_HIP, "%s: probe kernel launch failed: %s", fn,
                        hipGetErrorString(err));
    }
    const int64_t n_blocks = info->n_items > 0 ? slots * (info->tile / 32) : 0;
    hipLaunchKernelGGL(probe_reduce_kernel, dim3((unsigned)((hq * 3 + 3) / 4)), dim3(256), 0,
                       stream, part, n_blocks, hq * 3, region_sums);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess)
        return fail(TA_ERR_HIP, "%s: reduce kernel launch failed: %s", fn,
                    hipGetErrorString(err));
    return TA_OK;
}

extern "C" ta_status ta_region_counts(const int32_t *cu_seqlens, int32_t batch, int32_t sink,
                                      int32_t window, int32_t last, int64_t *counts)
{
    clear_error();
    static const char fn[] = "ta_region_counts";
    if (!cu_seqlens || !counts)
        return fail(TA_ERR_INVALID_ARG, "%s: cu_seqlens or counts is NULL", fn);
    if (batch < 0 || sink < 0 || window < 0 || last < 0)
        return fail(TA_ERR_INVALID_ARG, "%s: need batch, sink, window, last >= 0", fn);
    if (cu_seqlens[0] != 0)
        return fail(TA_ERR_INVALID_ARG, "%s: cu_seqlens[0] != 0", fn);
    int64_t c[3] = {0, 0, 0};
    for (int32_t b = 0; b < batch; ++b) {
        const int64_t n = (int64_t)cu_seqlens[b + 1] - cu_seqlens[b];
        if (n < 0)
            return fail(TA_ERR_INVALID_ARG, "%s: cu_seqlens decreases at %d", fn, b);
        const int64_t first_last = n - std::min<int64_t>(last, n);
        for (int64_t i = 0; i < n; ++i) {
            // row i: keys 0..i; window keys i - W + 1 .. i; sink keys below
            // the window
            const int64_t win = std::min<int64_t>(i + 1, window);
            const int64_t snk = std::min<int64_t>(sink, std::max<int64_t>(0, i - window + 1));
            c[0] += win + snk;
            c[i >= first_last ? 2 : 1] += i + 1 - win - snk;
        }
    }
    counts[0] = c[0];
    counts[1] = c[1];
    counts[2] = c[2];
    return TA_OK;
}

extern "C" ta_status ta_region_grad_mean(const double *region_sums, int32_t hq,
                                         const int64_t *counts, double *grad)
{
    clear_error();
    static const char fn[] = "ta_region_grad_mean";
    if (!region_sums || !counts || !grad)
        return fail(TA_ERR_INVALID_ARG, "%s: NULL argument", fn);
    if (hq <= 0)
        return fail(TA_ERR_INVALID_ARG, "%s: hq must be positive", fn);
    for (int r = 0; r < 3; ++r) {
        if (counts[r] < 0)
            return fail(TA_ERR_INVALID_ARG, "%s: negative count", fn);
        double s = 0.0;
        for (int32_t h = 0; h < hq; ++h)
            s += region_sums[h * 3 + r];
        grad[r] = counts[r] > 0 ? s / ((double)hq * (double)counts[r]) : 0.0;
    }
    return TA_OK;
}

extern "C" ta_status ta_select_triangle_layers(const double *grad_middle, int32_t n_layers,
                                               int32_t n_triangle, int32_t *layers)
{
    clear_error();
    static const char fn[] = "ta_select_triangle_layers";
    if (n_layers < 0 || n_triangle < 0 || n_triangle > n_layers)
        return fail(TA_ERR_INVALID_ARG, "%s: need 0 <= n_triangle <= n_layers", fn);
    if (n_layers > 0 && !grad_middle)
        return fail(TA_ERR_INVALID_ARG, "%s: grad_middle is NULL", fn);
    if (n_triangle > 0 && !layers)
        return fail(TA_ERR_INVALID_ARG, "%s: layers is NULL", fn);
    for (int32_t l = 0; l < n_layers; ++l)
        if (!std::isfinite(grad_middle[l]))
            return fail(TA_ERR_INVALID_ARG, "%s: grad_middle[%d] is not finite", fn, l);
    // the n_triangle layers whose middle section contributes least in
    // magnitude (ties: lower layer first), returned in increasing order
    std::vector<int32_t> order(n_layers);
    std::iota(order.begin(), order.end(), 0);
    std::stable_sort(order.begin(), order.end(), [&](int32_t x, int32_t y) {
        return std::fabs(grad_middle[x]) < std::fabs(grad_middle[y]);
    });
    order.resize(n_triangle);
    std::sort(order.begin(), order.end());
    std::copy(order.begin(), order.end(), layers);
    return TA_OK;
}
