// Internal declarations shared by the host schedule builder and the HIP
// forward passes of libtriattn.so.  Not part of the public interface.
#pragma once

#include <cstdint>
#include <cstdarg>

#include "triattn.h"

namespace triattn {

// Packed schedule layout (int32 words).
//   header (kHdrWords): magic, version, kind, tile, batch, sink, window, last,
//     splits requested, total_tokens low, total_tokens high, main items,
//     merge items, partial rows, kept k-tiles per query head, Last rows.
//   main item (kItemWords): seq_off, seq_len, r0, r1, ka0, ka1, kb0, kb1,
//     mode, part_base, kept k-tiles, 0.
//   merge item (kMergeWords): seq_off, r0, r1, splits, part_base, 0, 0, 0.
//   k-tile lists (block-sparse schedules only): int32 k-tile indices, after
//     the merge items; a list item (mode kModeCausalList) visits
//     lists[ka0 .. ka0 + ka1) in order.
constexpr int kHdrWords = 16;
constexpr int kItemWords = 12;
constexpr int kMergeWords = 8;

enum HdrField {
    H_MAGIC = 0, H_VERSION, H_KIND, H_TILE, H_BATCH, H_SINK, H_WINDOW, H_LAST,
    H_SPLITS, H_TOTAL_LO, H_TOTAL_HI, H_ITEMS, H_MERGES, H_PARTIAL_ROWS,
    H_KEPT_TILES, H_LAST_ROWS
};

enum ItemField {
    I_SEQ_OFF = 0, I_SEQ_LEN, I_R0, I_R1, I_KA0, I_KA1, I_KB0, I_KB1, I_MODE,
    I_PART_BASE, I_COST
};

enum MergeField { M_SEQ_OFF = 0, M_R0, M_R1, M_SPLITS, M_PART_BASE };

// Item masks: streaming rows keep j <= i && (j < sink || i - j < window);
// causal rows (Last rows, dense causal, block-sparse lists) keep j <= i.
constexpr int kModeStreaming = 0;
constexpr int kModeCausal = 1;
constexpr int kModeCausalList = 2;  // causal rows over a listed set of k-tiles

// Record a message for ta_last_error() and return the status.
ta_status fail(ta_status st, const char *fmt, ...);
void clear_error();

}  // namespace triattn
