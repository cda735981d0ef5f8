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
// Probe kernel: a workgroup owns one work item of a causal schedule (a q-tile
// and its k-tiles up to the diagonal), one kv head g and R rows of each of
// the G query heads of g, so every K/V tile staged in LDS serves the whole
// GQA group.  Each wave owns 32 rows of one head.  Per 64-key step it runs
// two bf16 MFMA 32x32x16 contractions with the same operand layout, S^T =
// K Q^T and dP^T = V dO^T (keys on the MFMA rows, queries on the columns), so
// a lane holds matching entries of both: it forms A = 2^(S c - lse log2 e)
// (c = scale log2 e; the row's LSE is an input, so no softmax state is
// carried) and adds A dP to the accumulator of the pair's section.  Per-step
// fp32 sums go into fp64 lane accumulators; each wave reduces them and writes
// one fp64 partial per (32-row block, head, section).  The reduce kernel sums
// the partials of each (head, section) in a fixed order, so results are
// deterministic.  Roofline: MFMA, 4 T^2 d flops per kept (q-tile, k-tile)
// pair and head, as the forward pass.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <numeric>
#include <vector>

#include "triattn_internal.h"

namespace triattn {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kProbeStep = 64;  // keys per step
constexpr float kProbeLog2e = 1.4426950408889634f;

struct ProbeArgs {
    const uint16_t *q;
    const uint16_t *k;
    const uint16_t *v;
    const uint16_t *dout;
    const float *lse;     // [hq, total] natural log
    const int32_t *sched;
    double *part;         // [n_items * tile / 32, hq, 3]
    int64_t total_tokens;
    int32_t hq, hkv, group;
    int32_t n_items;
    int32_t tile;
    int32_t rows_per_wg;  // R
    int32_t subtiles;     // tile / R
    int32_t sink, window, last;
    float scale_log2;     // softmax scale * log2(e)
};

// 16-byte chunk swizzle of LDS row r: the 32 rows one operand fetch reads
// land on distinct banks.
template <int D>
__device__ __forceinline__ int probe_swz(int r)
{
    return D == 128 ? (r & 15) : ((r >> 1) & 7);
}

__device__ __forceinline__ bool probe_header_ok(const int32_t *s, int64_t total,
                                                int32_t n_items, int32_t tile)
{
    const int64_t t = (int64_t)(uint32_t)s[H_TOTAL_LO] | ((int64_t)s[H_TOTAL_HI] << 32);
    return s[H_MAGIC] == TA_SCHEDULE_MAGIC && s[H_VERSION] == TA_SCHEDULE_VERSION &&
           s[H_KIND] == TA_KIND_CAUSAL && s[H_TILE] == tile && t == total &&
           s[H_ITEMS] == n_items;
}

template <int D, int NW>
__global__ __launch_bounds__(NW * 64) void probe_kernel(ProbeArgs a)
{
    constexpr int CH = D / 8;                        // 16-byte chunks per row
    constexpr int TILE_BYTES = kProbeStep * D * 2;   // one bf16 K or V tile
    constexpr int STAGE_BYTES = 2 * TILE_BYTES;      // K then V
    constexpr int CHUNKS = 2 * kProbeStep * CH;      // chunks per stage
    constexpr int NT = NW * 64;
    constexpr int CPT = (CHUNKS + NT - 1) / NT;      // chunks per thread
    constexpr int QK = D / 16;                       // MFMA k-steps over d
    __shared__ __attribute__((aligned(16))) uint8_t lds[2 * STAGE_BYTES];

    const int per_item = a.subtiles * a.hkv;
    const int item = blockIdx.x / per_item;
    const int rem = blockIdx.x - item * per_item;
    const int g = rem / a.subtiles;
    const int sub = rem - g * a.subtiles;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int h = lane >> 5;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wph = a.rows_per_wg / 32;  // waves per head
    const int head = g * a.group + wave / wph;
    const int rb = sub * wph + wave % wph;  // 32-row block within the q-tile

    double acc_s = 0.0, acc_o = 0.0;  // streaming / other (middle or last)
    bool last_row = false;

    const int32_t *sched = a.sched;
    bool ok = probe_header_ok(sched, a.total_tokens, a.n_items, a.tile);
    int64_t seq_off = 0;
    int32_t seq_len = 0, r0 = 0, r1 = 0, ka0 = 0, ka1 = 0;
    if (ok) {
        const int32_t *it = sched + kHdrWords + (int64_t)item * kItemWords;
        seq_off = it[I_SEQ_OFF];
        seq_len = it[I_SEQ_LEN];
        r0 = it[I_R0];
        r1 = it[I_R1];
        ka0 = it[I_KA0];
        ka1 = it[I_KA1];
        // guard against a malformed schedule: never touch memory outside it
        ok = it[I_MODE] == kModeCausal && it[I_KB0] == it[I_KB1] && seq_off >= 0 &&
             seq_len > 0 && seq_off + seq_len <= a.total_tokens && r0 >= 0 && r0 < r1 &&
             r1 <= seq_len && ka0 >= 0 && ka1 >= ka0;
    }
    const int wr0 = r0 + sub * a.rows_per_wg;  // first row of this workgroup
    ok = ok && wr0 < r1;                       // uniform over the workgroup

    if (ok) {
        const int row_base = wr0 + (wave % wph) * 32;
        const int my_row = row_base + (lane & 31);
        const bool row_valid = my_row < r1;
        const int load_row = row_valid ? my_row : r1 - 1;
        last_row = my_row >= seq_len - min(a.last, seq_len);
        const float c = a.scale_log2;
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

        // keys past the workgroup's last row are masked for all its rows
        const int wg_last = min(wr0 + a.rows_per_wg, r1) - 1;
        const int key_begin = ka0 * a.tile;
        const int key_end = min(ka1 * a.tile, wg_last + 1);
        const int nsteps = key_end > key_begin ? (key_end - key_begin + kProbeStep - 1) / kProbeStep : 0;

        // K/V staging: chunk x of a stage is tensor x / (64 CH) (0 = K, 1 =
        // V), row (x / CH) % 64, chunk column x % CH; rows past the
        // sequence repeat its last key (those keys are masked).
        u32x4 pf[CPT];
        auto load_step = [&](int s) {
            const int key0 = key_begin + s * kProbeStep;
#pragma unroll
            for (int i = 0; i < CPT; ++i) {
                const int x = tid + i * NT;
                if (CHUNKS % NT == 0 || x < CHUNKS) {
                    const int tensor = x / (kProbeStep * CH);
                    const int row = (x / CH) % kProbeStep;
                    const int col = x % CH;
                    const int key = min(key0 + row, seq_len - 1);
                    const uint16_t *src = (tensor ? a.v : a.k) +
                                          ((seq_off + key) * a.hkv + g) * (int64_t)D + col * 8;
                    pf[i] = *reinterpret_cast<const u32x4 *>(src);
                }
            }
        };
        auto store_step = [&](int stage) {
#pragma unroll
            for (int i = 0; i < CPT; ++i) {
                const int x = tid + i * NT;
                if (CHUNKS % NT == 0 || x < CHUNKS) {
                    const int tensor = x / (kProbeStep * CH);
                    const int row = (x / CH) % kProbeStep;
                    const int col = x % CH;
                    uint8_t *dst = lds + stage * STAGE_BYTES + tensor * TILE_BYTES +
                                   row * (D * 2) + ((col ^ probe_swz<D>(row)) << 4);
                    *reinterpret_cast<u32x4 *>(dst) = pf[i];
                }
            }
        };

        auto compute = [&](const uint8_t *st, int key0) {
            f32x16 sacc[2], gacc[2];
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) {
                const int r = kb * 32 + (lane & 31);
                const uint8_t *krow = st + r * (D * 2);
                const uint8_t *vrow = st + TILE_BYTES + r * (D * 2);
#pragma unroll
                for (int e = 0; e < 16; ++e) {
                    sacc[kb][e] = 0.f;
                    gacc[kb][e] = 0.f;
                }
#pragma unroll
                for (int s = 0; s < QK; ++s) {
                    const int off = ((2 * s + h) ^ probe_swz<D>(r)) << 4;
                    const bf16x8 kf = *reinterpret_cast<const bf16x8 *>(krow + off);
                    const bf16x8 vf = *reinterpret_cast<const bf16x8 *>(vrow + off);
                    sacc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[s], sacc[kb], 0, 0, 0);
                    gacc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, df[s], gacc[kb], 0, 0, 0);
                }
            }
            // register e of lane half h holds key key0 + 32 kb + (e & 3) +
            // 4 h + 8 (e >> 2) of this lane's row
            const bool all_causal = key0 + kProbeStep - 1 <= row_base && row_base + 31 < r1;
            const bool no_stream = key0 >= a.sink && row_base - (key0 + kProbeStep - 1) >= a.window;
            float ss = 0.f, so = 0.f;
            if (all_causal && no_stream) {
#pragma unroll
                for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                    for (int e = 0; e < 16; ++e)
                        so += __builtin_amdgcn_exp2f(fmaf(sacc[kb][e], c, -lse2)) * gacc[kb][e];
            } else {
#pragma unroll
                for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                    for (int e = 0; e < 16; ++e) {
                        const int key = key0 + 32 * kb + (e & 3) + 4 * h + 8 * (e >> 2);
                        const float p =
                            __builtin_amdgcn_exp2f(fmaf(sacc[kb][e], c, -lse2)) * gacc[kb][e];
                        const bool valid = row_valid && key <= my_row;
                        const bool strm = key < a.sink || my_row - key < a.window;
                        ss += (valid && strm) ? p : 0.f;
                        so += (valid && !strm) ? p : 0.f;
                    }
            }
            acc_s += (double)ss;
            acc_o += (double)so;
        };

        if (nsteps > 0) {
            load_step(0);
            store_step(0);
            if (nsteps > 1)
                load_step(1);
            __syncthreads();
            for (int s = 0; s < nsteps; ++s) {
                compute(lds + (s & 1) * STAGE_BYTES, key_begin + s * kProbeStep);
                if (s + 1 < nsteps) {
                    // stage (s + 1) & 1 was last read in step s - 1, before
                    // the barrier that ended it
                    store_step((s + 1) & 1);
                    if (s + 2 < nsteps)
                        load_step(s + 2);
                }
                __syncthreads();
            }
        }
    }

    double acc_m = last_row ? 0.0 : acc_o;
    double acc_l = last_row ? acc_o : 0.0;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
        acc_s += __shfl_xor(acc_s, off);
        acc_m += __shfl_xor(acc_m, off);
        acc_l += __shfl_xor(acc_l, off);
    }
    if (lane == 0) {
        // every partial is written (zero for rows past the q-tile), so the
        // workspace needs no clearing
        double *p = a.part + (((int64_t)item * (a.tile / 32) + rb) * a.hq + head) * 3;
        p[0] = acc_s;
        p[1] = acc_m;
        p[2] = acc_l;
    }
}

// out[hr] = sum over blocks b of part[b, hr] (hr = head * 3 + section), in a
// fixed order: thread-strided sums, then a tree over the workgroup.
__global__ __launch_bounds__(256) void probe_reduce_kernel(const double *part, int64_t n_blocks,
                                                           int32_t hq3, double *out)
{
    __shared__ double red[256];
    const int hr = blockIdx.x;
    double s = 0.0;
    for (int64_t b = threadIdx.x; b < n_blocks; b += 256)
        s += part[b * hq3 + hr];
    red[threadIdx.x] = s;
    __syncthreads();
    for (int w = 128; w > 0; w >>= 1) {
        if ((int)threadIdx.x < w)
            red[threadIdx.x] += red[threadIdx.x + w];
        __syncthreads();
    }
    if (threadIdx.x == 0)
        out[hr] = red[0];
}

int probe_rows_per_wg(int group, int tile)
{
    for (int r = 128; r >= 32; r /= 2)
        if (r <= tile && group * r / 32 <= 8)
            return r;
    return 32;
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
    return (size_t)info->n_items * (size_t)(info->tile / 32) * (size_t)hq * 3 * sizeof(double);
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
    if ((int64_t)info->n_items * subtiles * hkv > INT32_MAX)
        return fail(TA_ERR_UNSUPPORTED, "%s: grid too large", fn);

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
        const int nw = group * R / 32;
        dim3 grid((unsigned)((int64_t)info->n_items * subtiles * hkv));
        hipError_t err = head_dim == 128 ? launch_probe<128>(nw, grid, a, stream)
                                         : launch_probe<64>(nw, grid, a, stream);
        if (err != hipSuccess)
            return fail(TA_ERR_HIP, "%s: probe kernel launch failed: %s", fn,
                        hipGetErrorString(err));
    }
    const int64_t n_blocks = info->n_items > 0 ? (int64_t)info->n_items * (info->tile / 32) : 0;
    hipLaunchKernelGGL(probe_reduce_kernel, dim3((unsigned)(hq * 3)), dim3(256), 0, stream,
                       part, n_blocks, hq * 3, region_sums);
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
